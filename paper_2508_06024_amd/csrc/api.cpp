// C ABI of the EC2MoE hot path (declarations and contracts in include/ec2moe.h).
//
// Every entry point validates its arguments on the host first; on any error it returns
// before the first HIP call, so nothing is launched and no output is written. The error
// detail is kept per thread for ec2moe_last_error().
#include "ec2moe.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "internal.h"

namespace ec2moe {
namespace {

thread_local std::string g_last_error;

ec2moe_status fail(ec2moe_status st, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return st;
}

ec2moe_status ok() {
    g_last_error.clear();
    return EC2MOE_OK;
}

}  // namespace

ec2moe_status report_error(ec2moe_status st, const char* detail) {
    if (st == EC2MOE_OK) return ok();
    g_last_error = detail;
    return st;
}

namespace {

ec2moe_status hip_status(hipError_t e, const char* what) {
    if (e == hipSuccess) return ok();
    return fail(EC2MOE_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

#define REQUIRE(cond, st, ...) \
    do {                       \
        if (!(cond)) return fail(st, __VA_ARGS__); \
    } while (0)

#define REQUIRE_PTR(p) REQUIRE((p) != nullptr, EC2MOE_ERR_INVALID_ARGUMENT, "%s is NULL", #p)
#define REQUIRE_ALIGNED(p) REQUIRE(aligned16(p), EC2MOE_ERR_INVALID_ARGUMENT, "%s is not 16-byte aligned", #p)

constexpr int kMaxExperts = 256;
constexpr int kMaxGateRows = 320;
constexpr int kMaxTopK = 16;

// equal_groups: K must divide M (the gate without group sizes; the entry points after the
// gate never read the group structure)
ec2moe_status check_moe_desc(const ec2moe_moe_desc* d, bool equal_groups = true) {
    REQUIRE(d != nullptr, EC2MOE_ERR_INVALID_ARGUMENT, "desc is NULL");
    REQUIRE(d->dtype == EC2MOE_F32 || d->dtype == EC2MOE_BF16, EC2MOE_ERR_INVALID_ARGUMENT, "unknown dtype %d",
            static_cast<int>(d->dtype));
    REQUIRE(d->n_tokens >= 0, EC2MOE_ERR_INVALID_ARGUMENT, "n_tokens %d < 0", d->n_tokens);
    REQUIRE(d->n_experts > 0 && d->n_groups > 0 && d->d_model > 0 && d->ffn_hidden > 0 && d->top_k > 0,
            EC2MOE_ERR_INVALID_ARGUMENT, "n_experts, n_groups, d_model, ffn_hidden and top_k must be positive");
    REQUIRE(!equal_groups || d->n_experts % d->n_groups == 0, EC2MOE_ERR_INVALID_ARGUMENT,
            "n_groups %d does not divide n_experts %d", d->n_groups, d->n_experts);
    REQUIRE(d->n_groups <= d->n_experts, EC2MOE_ERR_INVALID_ARGUMENT, "n_groups %d > n_experts %d", d->n_groups,
            d->n_experts);
    REQUIRE(d->top_k <= d->n_experts, EC2MOE_ERR_INVALID_ARGUMENT, "top_k %d > n_experts %d", d->top_k,
            d->n_experts);
    REQUIRE((d->flags & ~(EC2MOE_GATE_RENORMALIZE | EC2MOE_EXPERT_RELU)) == 0, EC2MOE_ERR_INVALID_ARGUMENT,
            "unknown flags 0x%x", d->flags);
    REQUIRE(d->n_experts <= kMaxExperts, EC2MOE_ERR_UNSUPPORTED, "n_experts %d > %d", d->n_experts, kMaxExperts);
    REQUIRE(d->n_experts + d->n_groups <= kMaxGateRows, EC2MOE_ERR_UNSUPPORTED, "n_experts + n_groups > %d",
            kMaxGateRows);
    REQUIRE(d->top_k <= kMaxTopK, EC2MOE_ERR_UNSUPPORTED, "top_k %d > %d", d->top_k, kMaxTopK);
    REQUIRE(d->d_model % 128 == 0, EC2MOE_ERR_UNSUPPORTED, "d_model %d is not a multiple of 128", d->d_model);
    REQUIRE(d->ffn_hidden % 128 == 0, EC2MOE_ERR_UNSUPPORTED, "ffn_hidden %d is not a multiple of 128",
            d->ffn_hidden);
    // 32-bit byte offsets inside one operand of the GEMM
    const int64_t A = static_cast<int64_t>(d->n_tokens) * d->top_k;
    const int64_t eb = d->dtype == EC2MOE_F32 ? 4 : 2;
    REQUIRE(A * std::max(d->d_model, d->ffn_hidden) * eb < (int64_t(1) << 32) &&
                int64_t(2) * d->ffn_hidden * d->d_model * eb < (int64_t(1) << 32),
            EC2MOE_ERR_UNSUPPORTED, "tensor too large for 32-bit byte offsets");
    return EC2MOE_OK;
}

// ---------------------------------------------------------------- workspace carving
constexpr size_t kAlign = 256;
size_t up(size_t n) { return (n + kAlign - 1) / kAlign * kAlign; }

struct MoeWs {
    size_t counts, seg, perm_src, inv_perm, act, y_perm, part, total;
};

// split-K tail chunks of the large-tile GEMM
constexpr int kMaxSplit = 32;

MoeWs moe_ws(const ec2moe_moe_desc* d) {
    const int64_t A = static_cast<int64_t>(d->n_tokens) * d->top_k;
    const size_t eb = elem_bytes(static_cast<DType>(d->dtype));
    MoeWs w{};
    size_t o = 0;
    w.counts = o; o += up(static_cast<size_t>(std::max(1, perm_chunks(A))) * d->n_experts * 4);
    w.seg = o; o += up(static_cast<size_t>(d->n_experts + 1) * 4);
    w.perm_src = o; o += up(static_cast<size_t>(A) * 4);
    w.inv_perm = o; o += up(static_cast<size_t>(A) * 4);
    w.act = o; o += up(static_cast<size_t>(A) * d->ffn_hidden * eb);
    w.y_perm = o; o += up(static_cast<size_t>(A) * d->d_model * eb);
    w.part = o; o += up(gemm_split_scratch_bytes());
    w.total = o;
    return w;
}

template <typename T>
T* at(void* ws, size_t off) {
    return reinterpret_cast<T*>(static_cast<char*>(ws) + off);
}

ec2moe_status check_ws(void* ws, size_t have, size_t need) {
    REQUIRE(have >= need, EC2MOE_ERR_WORKSPACE_TOO_SMALL, "workspace of %zu bytes, %zu needed", have, need);
    REQUIRE(need == 0 || ws != nullptr, EC2MOE_ERR_INVALID_ARGUMENT, "ws is NULL");
    REQUIRE(aligned16(ws), EC2MOE_ERR_INVALID_ARGUMENT, "ws is not 16-byte aligned");
    return EC2MOE_OK;
}

// ---------------------------------------------------------------- codec plan
ec2moe_status check_codec_desc(const ec2moe_codec_desc* d) {
    REQUIRE(d != nullptr, EC2MOE_ERR_INVALID_ARGUMENT, "desc is NULL");
    REQUIRE(d->dtype == EC2MOE_F32 || d->dtype == EC2MOE_BF16, EC2MOE_ERR_INVALID_ARGUMENT, "unknown dtype %d",
            static_cast<int>(d->dtype));
    REQUIRE(d->n_slices >= 0 && d->h >= 0, EC2MOE_ERR_INVALID_ARGUMENT, "n_slices and h must be >= 0");
    REQUIRE(d->w > 0 && d->r_h > 0 && d->r_w > 0, EC2MOE_ERR_INVALID_ARGUMENT, "w, r_h and r_w must be positive");
    REQUIRE(d->r_h <= d->h || d->h == 0, EC2MOE_ERR_INVALID_ARGUMENT, "r_h %d > h %d", d->r_h, d->h);
    REQUIRE(d->r_w <= d->w, EC2MOE_ERR_INVALID_ARGUMENT, "r_w %d > w %d", d->r_w, d->w);
    REQUIRE(d->w % 128 == 0, EC2MOE_ERR_UNSUPPORTED, "w %d is not a multiple of 128", d->w);
    REQUIRE(d->r_h % 16 == 0 && d->r_w % 16 == 0 && d->r_h <= 256 && d->r_w <= 256, EC2MOE_ERR_UNSUPPORTED,
            "r_h and r_w must be multiples of 16 and at most 256");
    REQUIRE(static_cast<int64_t>(d->h) * d->w * (d->dtype == EC2MOE_F32 ? 4 : 2) < (int64_t(1) << 32),
            EC2MOE_ERR_UNSUPPORTED, "slice too large for 32-bit byte offsets");
    return EC2MOE_OK;
}

struct CodecWs {
    size_t gpart;  // split-K tail scratch of the matrix-core GEMMs (shared by encode and decode)
    int batch;     // slices handled by one set of launches
    // encode: V^T, P = X V (float32), per-chunk partial sums of U^T P
    size_t vt, p, epart, enc_total;
    int tc;      // tokens per chunk of the U^T P contraction
    bool fused;  // bf16 layers of whole 64-token and 64-column tiles: P and U^T P in one kernel
    bool small;  // at most 64 tokens per slice: the small-batch encoder and decoder
    // decode: Z rounded to the layer dtype (bf16 only), W = V_hat Z^T per slice, and the segment
    // offsets and row maps of the grouped products over a batch of slices
    size_t zb, wt, seg_w, rows_w, seg_h, rows_h, dec_total;
};

// Slices coded by one set of launches: at most 16, and few enough that a batch of X stays
// below 4 GiB (32-bit byte offsets in the GEMM's buffer descriptors).
constexpr int kMaxCodecBatch = 16;
int codec_batch(const ec2moe_codec_desc* d) {
    const int64_t slice = std::max<int64_t>(1, static_cast<int64_t>(d->h) * d->w * elem_bytes(static_cast<DType>(d->dtype)));
    const int64_t fit = ((int64_t(1) << 32) - 1) / slice;
    return static_cast<int>(std::max<int64_t>(1, std::min<int64_t>({fit, kMaxCodecBatch, std::max(1, d->n_slices)})));
}

// Token chunk of the U^T P contraction over (slice, chunk, 64-column block) workgroups:
// bfloat16 layers (three bf16 products per float32 one, about 1/5 of the float32 matrix-core
// time) aim at 128 workgroups of whole 64-token stages, halving the partial sums; float32
// layers at one workgroup per CU, in multiples of 4 tokens.
int utp_chunk(int h, int r_w, int slices, DType dt) {
    const int col_blocks = (r_w + 63) / 64;
    const bool bf16 = dt == DType::BF16;
    const int target = std::max(1, (bf16 ? 128 : 256) / (col_blocks * slices));
    const int tc = (std::max(1, h) + target - 1) / target;
    return bf16 ? (tc + 63) & ~63 : (tc + 3) & ~3;
}

CodecWs codec_ws(const ec2moe_codec_desc* d) {
    const size_t eb = elem_bytes(static_cast<DType>(d->dtype));
    CodecWs w{};
    w.batch = codec_batch(d);
    const size_t nb = static_cast<size_t>(w.batch);
    w.tc = utp_chunk(d->h, d->r_w, w.batch, static_cast<DType>(d->dtype));
    w.small = codec_small_ok(d->h, d->w, d->r_h, d->r_w);
    w.fused = !w.small && encode_fused_ok(static_cast<DType>(d->dtype), d->h, d->w, d->r_h, d->r_w);
    // partial sums of U^T P: per token chunk, or per 64-token tile of the fused encoder
    const size_t chunks = w.fused ? static_cast<size_t>(d->h) / 64
                                  : (static_cast<size_t>(std::max(1, d->h)) + w.tc - 1) / w.tc;
    size_t o = 0;
    w.gpart = o; o += up(gemm_split_scratch_bytes());
    const size_t shared = o;
    w.vt = o; o += w.fused ? 0 : up(static_cast<size_t>(d->r_w) * d->w * eb);  // the fused encoder reads V as stored
    w.p = o; o += w.fused || w.small ? 0 : up(nb * d->h * d->r_w * 4);
    w.epart = o;
    o += w.small ? up(codec_small_part_floats(d->h, d->w, d->r_w, static_cast<int>(nb)) * 4)
                 : up(nb * chunks * d->r_h * d->r_w * 4);
    w.enc_total = o;
    o = shared;
    // Z rounded to bf16 ahead of the decoder's GEMM, where the one-launch product does not apply
    const bool vzt = vzt_ok(static_cast<DType>(d->dtype), d->w, d->r_h, d->r_w);
    w.zb = o; o += vzt ? 0 : up(nb * d->r_h * d->r_w * eb);
    w.wt = o; o += up(nb * d->w * d->r_h * eb);
    w.seg_w = o; o += up((nb + 1) * 4);
    w.rows_w = o; o += up(nb * d->w * 4);
    w.seg_h = o; o += up((nb + 1) * 4);
    w.rows_h = o; o += up(nb * std::max(1, d->h) * 4);
    w.dec_total = o;
    return w;
}

// ---------------------------------------------------------------- kernel timing
struct ProfRecord {
    int name_id;
    hipEvent_t start, stop;
};

struct Profiler {
    std::mutex mu;
    bool enabled = false;
    std::string only;  // record only kernels of this name (empty: all)
    std::vector<std::string> names;
    std::vector<ProfRecord> records;
    std::vector<hipEvent_t> pool;

    int name_id(const char* n) {
        for (size_t i = 0; i < names.size(); ++i)
            if (names[i] == n) return static_cast<int>(i);
        names.emplace_back(n);
        return static_cast<int>(names.size() - 1);
    }
    hipEvent_t get() {
        if (!pool.empty()) {
            hipEvent_t e = pool.back();
            pool.pop_back();
            return e;
        }
        // Timing-only events, without the system-scope fence of a default event record (a
        // writeback of every XCD's L2). An event record still leaves ~5 us of idle time on
        // each side of a timed kernel (layer step: 2.544 against 2.538 ms per step untimed).
        hipEvent_t e = nullptr;
        if (hipEventCreateWithFlags(&e, hipEventDisableSystemFence) != hipSuccess) return nullptr;
        return e;
    }
};

Profiler& prof() {
    static Profiler p;
    return p;
}

}  // namespace

ProfileScope::ProfileScope(const char* name, hipStream_t s) : slot(-1), stream(s) {
    Profiler& p = prof();
    std::lock_guard<std::mutex> lk(p.mu);
    if (!p.enabled || (!p.only.empty() && p.only != name)) return;
    ProfRecord r{p.name_id(name), p.get(), p.get()};
    if (!r.start || !r.stop) return;
    if (hipEventRecord(r.start, s) != hipSuccess) return;
    p.records.push_back(r);
    slot = static_cast<int>(p.records.size() - 1);
}

ProfileScope::~ProfileScope() {
    if (slot < 0) return;
    Profiler& p = prof();
    std::lock_guard<std::mutex> lk(p.mu);
    if (slot < static_cast<int>(p.records.size())) (void)hipEventRecord(p.records[slot].stop, stream);
}

}  // namespace ec2moe

using namespace ec2moe;

extern "C" {

const char* ec2moe_status_string(ec2moe_status s) {
    switch (s) {
        case EC2MOE_OK: return "ok";
        case EC2MOE_ERR_INVALID_ARGUMENT: return "invalid argument";
        case EC2MOE_ERR_UNSUPPORTED: return "unsupported shape or type";
        case EC2MOE_ERR_TOO_FEW_CANDIDATES: return "fewer candidate experts than top_k";
        case EC2MOE_ERR_WORKSPACE_TOO_SMALL: return "workspace too small";
        case EC2MOE_ERR_HIP: return "HIP error";
    }
    return "unknown status";
}

const char* ec2moe_last_error(void) { return g_last_error.c_str(); }

ec2moe_status ec2moe_group_gate_ex(const ec2moe_moe_desc* desc, const ec2moe_gate_opts* opts,
                                   const uint64_t* cand_mask, const void* x, const void* w_global,
                                   const float* b_global, const void* w_local, const float* b_local,
                                   int32_t* topk_idx, float* topk_w, float* probs, hipStream_t stream) {
    const bool sized = opts && opts->group_sizes;
    if (ec2moe_status st = check_moe_desc(desc, !sized); st != EC2MOE_OK) return st;
    REQUIRE_PTR(cand_mask);
    const int M = desc->n_experts, K = desc->n_groups;
    const int top_groups = opts ? opts->top_groups : 0;
    REQUIRE(top_groups >= 0, EC2MOE_ERR_INVALID_ARGUMENT, "top_groups %d < 0", top_groups);
    GateArgs a{};
    a.top_groups = top_groups;
    a.equal_groups = sized ? 0 : 1;
    a.goff[0] = 0;
    for (int k = 0; k < K; ++k) {
        const int mk = sized ? opts->group_sizes[k] : M / K;
        REQUIRE(mk >= 1, EC2MOE_ERR_INVALID_ARGUMENT, "group %d has %d experts", k, mk);
        a.goff[k + 1] = a.goff[k] + mk;
        REQUIRE(a.goff[k + 1] <= M, EC2MOE_ERR_INVALID_ARGUMENT, "group sizes exceed n_experts %d", M);
    }
    REQUIRE(a.goff[K] == M, EC2MOE_ERR_INVALID_ARGUMENT, "group sizes sum to %d, not n_experts %d", a.goff[K], M);
    const int words = (M + 63) / 64;
    int pop = 0;
    for (int i = 0; i < words; ++i) {
        uint64_t v = cand_mask[i];
        const int valid_bits = std::min(64, M - 64 * i);
        if (valid_bits < 64) REQUIRE((v >> valid_bits) == 0, EC2MOE_ERR_INVALID_ARGUMENT,
                                     "cand_mask has bits set at or above n_experts %d", M);
        pop += __builtin_popcountll(v);
    }
    REQUIRE(pop >= desc->top_k, EC2MOE_ERR_TOO_FEW_CANDIDATES, "%d candidate experts for top-%d", pop,
            desc->top_k);
    if (desc->n_tokens == 0) return ok();
    REQUIRE_PTR(x); REQUIRE_PTR(w_global); REQUIRE_PTR(w_local); REQUIRE_PTR(topk_idx); REQUIRE_PTR(topk_w);
    REQUIRE_ALIGNED(x); REQUIRE_ALIGNED(w_global); REQUIRE_ALIGNED(w_local);
    a.x = x; a.w_global = w_global; a.b_global = b_global; a.w_local = w_local; a.b_local = b_local;
    a.topk_idx = topk_idx; a.topk_w = topk_w; a.probs = probs;
    a.n_tokens = desc->n_tokens; a.d = desc->d_model; a.n_experts = M; a.n_groups = K;
    a.top_k = desc->top_k; a.renormalize = (desc->flags & EC2MOE_GATE_RENORMALIZE) != 0;
    for (int i = 0; i < 4; ++i) a.mask[i] = i < words ? cand_mask[i] : 0;
    const DType dt = static_cast<DType>(desc->dtype);
    if (opts && opts->workspace) {
        const size_t need = gate_split_bytes(dt, desc->n_tokens, desc->d_model, M + K);
        REQUIRE(opts->workspace_bytes >= need, EC2MOE_ERR_WORKSPACE_TOO_SMALL,
                "gate workspace of %zu bytes, %zu needed", opts->workspace_bytes, need);
        REQUIRE(aligned16(opts->workspace), EC2MOE_ERR_INVALID_ARGUMENT, "gate workspace is not 16-byte aligned");
        if (need > 0) {
            a.ws = static_cast<float*>(opts->workspace);
            a.nsplit = gate_split_count(dt, desc->n_tokens, desc->d_model);
        }
    }
    return hip_status(launch_gate(dt, a, stream), "gate launch");
}

ec2moe_status ec2moe_gate_workspace_size(const ec2moe_moe_desc* desc, size_t* bytes) {
    if (ec2moe_status st = check_moe_desc(desc, false); st != EC2MOE_OK) return st;
    REQUIRE_PTR(bytes);
    *bytes = gate_split_bytes(static_cast<DType>(desc->dtype), desc->n_tokens, desc->d_model,
                              desc->n_experts + desc->n_groups);
    return ok();
}

ec2moe_status ec2moe_group_gate(const ec2moe_moe_desc* desc, const uint64_t* cand_mask, const void* x,
                                const void* w_global, const float* b_global, const void* w_local,
                                const float* b_local, int32_t* topk_idx, float* topk_w, float* probs,
                                hipStream_t stream) {
    return ec2moe_group_gate_ex(desc, nullptr, cand_mask, x, w_global, b_global, w_local, b_local, topk_idx,
                                topk_w, probs, stream);
}

ec2moe_status ec2moe_moe_workspace_size(const ec2moe_moe_desc* desc, size_t* bytes) {
    if (ec2moe_status st = check_moe_desc(desc, false); st != EC2MOE_OK) return st;
    REQUIRE_PTR(bytes);
    *bytes = moe_ws(desc).total;
    return ok();
}

ec2moe_status ec2moe_permute(const ec2moe_moe_desc* desc, const int32_t* topk_idx, const void* x,
                             int32_t* seg_offsets, int32_t* perm_src, int32_t* inv_perm, void* x_perm, void* ws,
                             size_t ws_bytes, hipStream_t stream) {
    if (ec2moe_status st = check_moe_desc(desc, false); st != EC2MOE_OK) return st;
    const MoeWs w = moe_ws(desc);
    if (ec2moe_status st = check_ws(ws, ws_bytes, w.total); st != EC2MOE_OK) return st;
    REQUIRE_PTR(seg_offsets);
    REQUIRE((x == nullptr) == (x_perm == nullptr), EC2MOE_ERR_INVALID_ARGUMENT,
            "x and x_perm must both be given or both be NULL");
    const int64_t A = static_cast<int64_t>(desc->n_tokens) * desc->top_k;
    if (A > 0) {
        REQUIRE_PTR(topk_idx); REQUIRE_PTR(perm_src); REQUIRE_PTR(inv_perm);
        if (x) { REQUIRE_ALIGNED(x); REQUIRE_ALIGNED(x_perm); }
    }
    hipError_t e = launch_permute(topk_idx, A, desc->top_k, desc->n_experts, at<int32_t>(ws, w.counts),
                                  seg_offsets, perm_src, inv_perm, stream);
    if (e == hipSuccess && x)
        e = launch_gather_rows(static_cast<DType>(desc->dtype), x, desc->n_tokens, perm_src,
                               seg_offsets + desc->n_experts, A, desc->d_model, x_perm, stream);
    return hip_status(e, "permute launch");
}

ec2moe_status ec2moe_permute_noalloc(const ec2moe_moe_desc* desc, const int32_t* topk_idx, const void* x,
                                     int32_t* seg_offsets, int32_t* perm_src, int32_t* inv_perm, void* x_perm,
                                     hipStream_t stream) {
    if (ec2moe_status st = check_moe_desc(desc, false); st != EC2MOE_OK) return st;
    REQUIRE_PTR(seg_offsets);
    REQUIRE((x == nullptr) == (x_perm == nullptr), EC2MOE_ERR_INVALID_ARGUMENT,
            "x and x_perm must both be given or both be NULL");
    const int64_t A = static_cast<int64_t>(desc->n_tokens) * desc->top_k;
    const int64_t words = static_cast<int64_t>(perm_chunks(A)) * desc->n_experts;
    REQUIRE(words <= kPermStaticCountWords, EC2MOE_ERR_UNSUPPORTED,
            "%lld assignments over %d experts need %lld count words; the library's own array holds %d "
            "(ceil(T*k / %d) * n_experts <= %d): pass a workspace to ec2moe_permute instead",
            static_cast<long long>(A), desc->n_experts, static_cast<long long>(words), kPermStaticCountWords,
            kPermChunk, kPermStaticCountWords);
    if (A > 0) {
        REQUIRE_PTR(topk_idx); REQUIRE_PTR(perm_src); REQUIRE_PTR(inv_perm);
        if (x) { REQUIRE_ALIGNED(x); REQUIRE_ALIGNED(x_perm); }
    }
    int32_t* counts = nullptr;
    hipError_t e = permute_static_counts(&counts);
    if (e != hipSuccess) return hip_status(e, "permute_noalloc: device count array");
    e = launch_permute(topk_idx, A, desc->top_k, desc->n_experts, counts, seg_offsets, perm_src, inv_perm, stream);
    if (e == hipSuccess && x)
        e = launch_gather_rows(static_cast<DType>(desc->dtype), x, desc->n_tokens, perm_src,
                               seg_offsets + desc->n_experts, A, desc->d_model, x_perm, stream);
    return hip_status(e, "permute_noalloc launch");
}

namespace {

hipError_t run_experts(const ec2moe_moe_desc* desc, const void* x, const int32_t* seg, const int32_t* perm_src,
                       const void* w_gate_up, const void* w_down, void* act, void* y_perm, float* part,
                       hipStream_t stream) {
    const DType dt = static_cast<DType>(desc->dtype);
    const int64_t A = static_cast<int64_t>(desc->n_tokens) * desc->top_k;
    const int d = desc->d_model, H = desc->ffn_hidden;
    // SwiGLU: [2H][d] gate and up rows per expert; ReLU: [H][d] input-layer rows
    const bool relu = (desc->flags & EC2MOE_EXPERT_RELU) != 0;
    const int64_t w_in_rows = relu ? H : int64_t(2) * H;
    GemmArgs g1{};
    g1.tok = x; g1.row_index = perm_src; g1.w = w_gate_up;
    g1.w_group_stride = w_in_rows * d; g1.seg = seg; g1.n_groups = desc->n_experts;
    g1.rows = A; g1.K = d; g1.N = H; g1.out = act; g1.ldo = H; g1.name = relu ? "expert_in_relu" : "expert_gate_up";
    g1.src_rows = desc->n_tokens; g1.w_rows = w_in_rows; g1.part = part; g1.max_split = kMaxSplit;
    hipError_t e = launch_gemm(dt, relu ? Epilogue::ReLU : Epilogue::SwiGLU, OutType::Same, g1, stream);
    if (e != hipSuccess) return e;
    GemmArgs g2{};
    g2.tok = act; g2.row_index = nullptr; g2.w = w_down;
    g2.w_group_stride = int64_t(d) * H; g2.seg = seg; g2.n_groups = desc->n_experts;
    g2.rows = A; g2.K = H; g2.N = d; g2.out = y_perm; g2.ldo = d; g2.name = "expert_down";
    g2.src_rows = A; g2.w_rows = d; g2.part = part; g2.max_split = kMaxSplit;
    return launch_gemm(dt, Epilogue::Store, OutType::Same, g2, stream);
}

}  // namespace

ec2moe_status ec2moe_expert_ffn(const ec2moe_moe_desc* desc, const void* x, const int32_t* seg_offsets,
                                const int32_t* perm_src, const void* w_gate_up, const void* w_down, void* act,
                                void* y_perm, void* ws, size_t ws_bytes, hipStream_t stream) {
    if (ec2moe_status st = check_moe_desc(desc, false); st != EC2MOE_OK) return st;
    const MoeWs w = moe_ws(desc);
    if (ec2moe_status st = check_ws(ws, ws_bytes, w.total); st != EC2MOE_OK) return st;
    if (desc->n_tokens == 0) return ok();
    REQUIRE_PTR(x); REQUIRE_PTR(seg_offsets); REQUIRE_PTR(perm_src); REQUIRE_PTR(w_gate_up); REQUIRE_PTR(w_down);
    REQUIRE_PTR(y_perm);
    REQUIRE_ALIGNED(x); REQUIRE_ALIGNED(w_gate_up); REQUIRE_ALIGNED(w_down); REQUIRE_ALIGNED(y_perm);
    if (act) REQUIRE_ALIGNED(act);
    void* act_buf = act ? act : at<void>(ws, w.act);
    return hip_status(run_experts(desc, x, seg_offsets, perm_src, w_gate_up, w_down, act_buf, y_perm,
                                  at<float>(ws, w.part), stream),
                      "expert GEMM launch");
}

ec2moe_status ec2moe_combine(const ec2moe_moe_desc* desc, const void* y_perm, const int32_t* inv_perm,
                             const float* topk_w, void* y, hipStream_t stream) {
    if (ec2moe_status st = check_moe_desc(desc, false); st != EC2MOE_OK) return st;
    if (desc->n_tokens == 0) return ok();
    REQUIRE_PTR(y_perm); REQUIRE_PTR(inv_perm); REQUIRE_PTR(topk_w); REQUIRE_PTR(y);
    REQUIRE_ALIGNED(y_perm); REQUIRE_ALIGNED(y);
    return hip_status(launch_combine(static_cast<DType>(desc->dtype), y_perm, inv_perm, topk_w, desc->n_tokens,
                                     desc->top_k, desc->d_model, y, stream),
                      "combine launch");
}

ec2moe_status ec2moe_moe_forward(const ec2moe_moe_desc* desc, const void* x, const int32_t* topk_idx,
                                 const float* topk_w, const void* w_gate_up, const void* w_down, void* y, void* ws,
                                 size_t ws_bytes, hipStream_t stream) {
    if (ec2moe_status st = check_moe_desc(desc, false); st != EC2MOE_OK) return st;
    const MoeWs w = moe_ws(desc);
    if (ec2moe_status st = check_ws(ws, ws_bytes, w.total); st != EC2MOE_OK) return st;
    if (desc->n_tokens == 0) return ok();
    REQUIRE_PTR(x); REQUIRE_PTR(topk_idx); REQUIRE_PTR(topk_w); REQUIRE_PTR(w_gate_up); REQUIRE_PTR(w_down);
    REQUIRE_PTR(y);
    REQUIRE_ALIGNED(x); REQUIRE_ALIGNED(w_gate_up); REQUIRE_ALIGNED(w_down); REQUIRE_ALIGNED(y);
    const int64_t A = static_cast<int64_t>(desc->n_tokens) * desc->top_k;
    int32_t* seg = at<int32_t>(ws, w.seg);
    int32_t* perm_src = at<int32_t>(ws, w.perm_src);
    int32_t* inv_perm = at<int32_t>(ws, w.inv_perm);
    void* act = at<void>(ws, w.act);
    void* y_perm = at<void>(ws, w.y_perm);
    hipError_t e = launch_permute(topk_idx, A, desc->top_k, desc->n_experts, at<int32_t>(ws, w.counts), seg,
                                  perm_src, inv_perm, stream);
    if (e == hipSuccess)
        e = run_experts(desc, x, seg, perm_src, w_gate_up, w_down, act, y_perm, at<float>(ws, w.part), stream);
    if (e == hipSuccess)
        e = launch_combine(static_cast<DType>(desc->dtype), y_perm, inv_perm, topk_w, desc->n_tokens, desc->top_k,
                           desc->d_model, y, stream);
    return hip_status(e, "moe_forward launch");
}

ec2moe_status ec2moe_lowrank_workspace_size(const ec2moe_codec_desc* desc, size_t* bytes) {
    if (ec2moe_status st = check_codec_desc(desc); st != EC2MOE_OK) return st;
    REQUIRE_PTR(bytes);
    const CodecWs w = codec_ws(desc);
    *bytes = std::max(w.enc_total, w.dec_total);
    return ok();
}

ec2moe_status ec2moe_lowrank_encode(const ec2moe_codec_desc* desc, const void* x, const void* u, const void* v,
                                    float* z, void* ws, size_t ws_bytes, hipStream_t stream) {
    if (ec2moe_status st = check_codec_desc(desc); st != EC2MOE_OK) return st;
    const CodecWs w = codec_ws(desc);
    if (ec2moe_status st = check_ws(ws, ws_bytes, std::max(w.enc_total, w.dec_total)); st != EC2MOE_OK) return st;
    if (desc->n_slices == 0) return ok();
    REQUIRE(desc->h > 0, EC2MOE_ERR_INVALID_ARGUMENT, "h must be positive");
    REQUIRE_PTR(x); REQUIRE_PTR(u); REQUIRE_PTR(v); REQUIRE_PTR(z);
    REQUIRE_ALIGNED(x); REQUIRE_ALIGNED(u); REQUIRE_ALIGNED(v); REQUIRE_ALIGNED(z);
    const DType dt = static_cast<DType>(desc->dtype);
    const size_t eb = elem_bytes(dt);
    const size_t slice_bytes = static_cast<size_t>(desc->h) * desc->w * eb;
    if (w.small) {
        hipError_t e = hipSuccess;
        for (int c0 = 0; c0 < desc->n_slices && e == hipSuccess; c0 += w.batch) {
            const int nc = std::min(w.batch, desc->n_slices - c0);
            e = launch_encode_small(dt, static_cast<const char*>(x) + c0 * slice_bytes, u, v, desc->h, desc->w,
                                    desc->r_h, desc->r_w, nc, at<float>(ws, w.epart),
                                    z + static_cast<size_t>(c0) * desc->r_h * desc->r_w, stream);
        }
        return hip_status(e, "lowrank_encode launch");
    }
    void* vt = at<void>(ws, w.vt);
    float* p = at<float>(ws, w.p);
    hipError_t e = w.fused ? hipSuccess : launch_transpose(dt, v, desc->w, desc->r_w, vt, stream);
    for (int c0 = 0; c0 < desc->n_slices && e == hipSuccess; c0 += w.batch) {
        const int nc = std::min(w.batch, desc->n_slices - c0);
        if (w.fused) {
            EncArgs a{};
            a.x = static_cast<const char*>(x) + c0 * slice_bytes; a.v = v; a.u = u; a.part = at<float>(ws, w.epart);
            a.h = desc->h; a.w = desc->w; a.rh = desc->r_h; a.rw = desc->r_w; a.slices = nc;
            e = launch_encode_fused(a, z + static_cast<size_t>(c0) * desc->r_h * desc->r_w, stream);
            continue;
        }
        // P = X V  [nc * h][r_w], float32: V is shared, so the slices stack into one product
        GemmArgs g{};
        g.tok = static_cast<const char*>(x) + c0 * slice_bytes; g.row_index = nullptr; g.w = vt;
        g.w_group_stride = 0; g.seg = nullptr; g.n_groups = 1;
        g.rows = int64_t(nc) * desc->h; g.K = desc->w; g.N = desc->r_w; g.out = p; g.ldo = desc->r_w;
        g.name = "codec_xv";
        g.src_rows = g.rows; g.w_rows = desc->r_w; g.part = at<float>(ws, w.gpart); g.max_split = kMaxSplit;
        e = launch_gemm(dt, Epilogue::Store, OutType::F32, g, stream);
        if (e != hipSuccess) break;
        // Z[s] = U^T P[s]  [r_h][r_w] per slice, float32 over token chunks, reduced in chunk order
        UtpArgs a{};
        a.u = u; a.p = p; a.T = desc->h; a.rh = desc->r_h; a.rw = desc->r_w; a.tc = w.tc; a.slices = nc;
        a.part = at<float>(ws, w.epart); a.z = z + static_cast<size_t>(c0) * desc->r_h * desc->r_w;
        e = launch_utp(dt, a, stream);
    }
    return hip_status(e, "lowrank_encode launch");
}

ec2moe_status ec2moe_lowrank_decode(const ec2moe_codec_desc* desc, const float* z, const void* u_hat,
                                    const void* v_hat, void* x_hat, void* ws, size_t ws_bytes, hipStream_t stream) {
    if (ec2moe_status st = check_codec_desc(desc); st != EC2MOE_OK) return st;
    const CodecWs w = codec_ws(desc);
    if (ec2moe_status st = check_ws(ws, ws_bytes, std::max(w.enc_total, w.dec_total)); st != EC2MOE_OK) return st;
    if (desc->n_slices == 0) return ok();
    REQUIRE(desc->h > 0, EC2MOE_ERR_INVALID_ARGUMENT, "h must be positive");
    REQUIRE_PTR(z); REQUIRE_PTR(u_hat); REQUIRE_PTR(v_hat); REQUIRE_PTR(x_hat);
    REQUIRE_ALIGNED(z); REQUIRE_ALIGNED(u_hat); REQUIRE_ALIGNED(v_hat); REQUIRE_ALIGNED(x_hat);
    const DType dt = static_cast<DType>(desc->dtype);
    const size_t eb = elem_bytes(dt);
    void* wt = at<void>(ws, w.wt);
    hipError_t e = hipSuccess;
    const int64_t zn = static_cast<int64_t>(desc->r_h) * desc->r_w;
    if (w.small) {
        const size_t slice_bytes = static_cast<size_t>(desc->h) * desc->w * eb;
        for (int c0 = 0; c0 < desc->n_slices && e == hipSuccess; c0 += w.batch) {
            const int nc = std::min(w.batch, desc->n_slices - c0);
            e = launch_decode_small(dt, z + static_cast<size_t>(c0) * zn, u_hat, v_hat, desc->h, desc->w, desc->r_h,
                                    desc->r_w, nc, static_cast<char*>(x_hat) + c0 * slice_bytes, stream);
        }
        return hip_status(e, "lowrank_decode launch");
    }
    if (desc->n_slices == 1) {
        // Wt = V_hat Z^T  [w][r_h]: both operands are K-contiguous rows (V_hat [w][r_w], Z [r_h][r_w]).
        // In bf16 layers Z is rounded to bf16 first (the product runs on the bf16 matrix cores;
        // Wt itself is rounded to bf16 anyway), inside the one-launch product where the shape allows.
        if (vzt_ok(dt, desc->w, desc->r_h, desc->r_w)) {
            e = launch_vzt(z, v_hat, desc->w, desc->r_h, desc->r_w, 1, wt, stream);
        } else {
            const void* zop = z;
            if (dt == DType::BF16) {
                e = launch_f32_to_bf16(z, zn, at<void>(ws, w.zb), stream);
                zop = at<void>(ws, w.zb);
            }
            if (e == hipSuccess) {
                GemmArgs gw{};
                gw.tok = v_hat; gw.row_index = nullptr; gw.w = zop; gw.w_group_stride = 0; gw.seg = nullptr;
                gw.n_groups = 1; gw.rows = desc->w; gw.K = desc->r_w; gw.N = desc->r_h; gw.out = wt; gw.ldo = desc->r_h;
                gw.name = "codec_vzt";
                gw.src_rows = desc->w; gw.w_rows = desc->r_h; gw.part = at<float>(ws, w.gpart); gw.max_split = kMaxSplit;
                e = launch_gemm(dt, Epilogue::Store, OutType::Same, gw, stream);
            }
        }
        if (e == hipSuccess && expand_ok(dt, desc->h, desc->w, desc->r_h)) {
            e = launch_expand(u_hat, wt, desc->h, desc->w, desc->r_h, x_hat, stream);
        } else if (e == hipSuccess) {
            // X_hat = U_hat Wt^T  [h][w]
            GemmArgs g{};
            g.tok = u_hat; g.row_index = nullptr; g.w = wt; g.w_group_stride = 0; g.seg = nullptr; g.n_groups = 1;
            g.rows = desc->h; g.K = desc->r_h; g.N = desc->w; g.out = x_hat; g.ldo = desc->w; g.name = "codec_uw";
            g.src_rows = desc->h; g.w_rows = desc->w; g.part = at<float>(ws, w.gpart); g.max_split = kMaxSplit;
            e = launch_gemm(dt, Epilogue::Store, OutType::Same, g, stream);
        }
        return hip_status(e, "lowrank_decode launch");
    }
    // Several slices: the same two products as grouped GEMMs with one group per slice of a
    // batch (the token-side operand V_hat or U_hat gathered through a row map p -> p mod rows).
    int32_t* seg_w = at<int32_t>(ws, w.seg_w);
    int32_t* rows_w = at<int32_t>(ws, w.rows_w);
    int32_t* seg_h = at<int32_t>(ws, w.seg_h);
    int32_t* rows_h = at<int32_t>(ws, w.rows_h);
    for (int c0 = 0; c0 < desc->n_slices && e == hipSuccess; c0 += w.batch) {
        const int nc = std::min(w.batch, desc->n_slices - c0);
        const float* zc = z + static_cast<size_t>(c0) * zn;
        const bool vzt = vzt_ok(dt, desc->w, desc->r_h, desc->r_w);
        void* zb = dt == DType::BF16 && !vzt ? at<void>(ws, w.zb) : nullptr;
        e = launch_codec_prep(zc, nc * zn, zb, nc, desc->w, desc->h, seg_w, rows_w, seg_h, rows_h, stream);
        if (e != hipSuccess) break;
        // Wt[s] = V_hat Z[s]^T  [w][r_h]
        if (vzt) {
            e = launch_vzt(zc, v_hat, desc->w, desc->r_h, desc->r_w, nc, wt, stream);
        } else {
            GemmArgs gw{};
            gw.tok = v_hat; gw.row_index = rows_w; gw.w = zb ? zb : static_cast<const void*>(zc);
            gw.w_group_stride = zn; gw.seg = seg_w; gw.n_groups = nc; gw.rows = int64_t(nc) * desc->w;
            gw.K = desc->r_w; gw.N = desc->r_h; gw.out = wt; gw.ldo = desc->r_h; gw.name = "codec_vzt";
            gw.src_rows = desc->w; gw.w_rows = desc->r_h; gw.part = at<float>(ws, w.gpart); gw.max_split = kMaxSplit;
            e = launch_gemm(dt, Epilogue::Store, OutType::Same, gw, stream);
        }
        if (e != hipSuccess) break;
        // X_hat[s] = U_hat Wt[s]^T  [h][w]
        GemmArgs g{};
        g.tok = u_hat; g.row_index = rows_h; g.w = wt; g.w_group_stride = int64_t(desc->w) * desc->r_h;
        g.seg = seg_h; g.n_groups = nc; g.rows = int64_t(nc) * desc->h; g.K = desc->r_h; g.N = desc->w;
        g.out = static_cast<char*>(x_hat) + static_cast<size_t>(c0) * desc->h * desc->w * eb; g.ldo = desc->w;
        g.name = "codec_uw";
        g.src_rows = desc->h; g.w_rows = desc->w; g.part = at<float>(ws, w.gpart); g.max_split = kMaxSplit;
        e = launch_gemm(dt, Epilogue::Store, OutType::Same, g, stream);
    }
    return hip_status(e, "lowrank_decode launch");
}

namespace {

struct FitWs {
    size_t gpart, gram, xt, q, y, q1, qt, g64, g64part, rinv_t, total;
};

FitWs fit_ws(const ec2moe_codec_desc* d) {
    const size_t eb = elem_bytes(static_cast<DType>(d->dtype));
    const size_t n = static_cast<size_t>(std::max(d->h, d->w));
    const size_t r = static_cast<size_t>(std::max(d->r_h, d->r_w));
    const size_t cells = static_cast<size_t>(std::max(1, d->n_slices)) * d->h * d->w;
    FitWs w{};
    size_t o = 0;
    w.gpart = o; o += up(gemm_split_scratch_bytes());
    w.gram = o; o += up(n * n * 4);
    w.xt = o; o += up(cells * eb);
    w.q = o; o += up(n * r * 4);
    w.y = o; o += up(n * r * 4);
    w.q1 = o; o += up(n * r * 4);
    w.qt = o; o += up(n * r * 4);
    w.g64 = o; o += up(r * r * 8);
    const int chunks = std::max(gram64_chunks(d->h, static_cast<int>(d->r_h)), gram64_chunks(d->w, static_cast<int>(d->r_w)));
    w.g64part = o; o += up(static_cast<size_t>(chunks) * r * r * 8);
    w.rinv_t = o; o += up(r * r * 4);
    w.total = o;
    return w;
}

hipError_t dense_gemm(DType dt, OutType ot, const void* tok, const void* wt, int64_t rows, int K, int N, void* out,
                      const char* name, float* part, hipStream_t s) {
    GemmArgs g{};
    g.tok = tok; g.row_index = nullptr; g.w = wt; g.w_group_stride = 0; g.seg = nullptr; g.n_groups = 1;
    g.rows = rows; g.K = K; g.N = N; g.out = out; g.ldo = N; g.name = name;
    g.src_rows = rows; g.w_rows = N; g.part = part; g.max_split = kMaxSplit;
    return launch_gemm(dt, Epilogue::Store, ot, g, s);
}

// Q = orth(Y) for Y [n][r] float32 (CholeskyQR2, the first pass into q1); q receives the result.
hipError_t orthonormalise(float* y, int n, int r, float* q1, float* q, const FitWs& w, void* ws, int32_t* status,
                          bool& reset, hipStream_t s) {
    double* g64 = at<double>(ws, w.g64);
    float* rinv_t = at<float>(ws, w.rinv_t);
    float* part = at<float>(ws, w.gpart);
    const float* src = y;
    for (int pass = 0; pass < 2; ++pass) {
        float* dst = pass == 0 ? q1 : q;
        hipError_t e = launch_gram64(src, n, r, at<double>(ws, w.g64part), g64, s);
        if (e == hipSuccess) e = launch_chol_inv(g64, r, rinv_t, status, reset, s);
        reset = false;
        if (e == hipSuccess) e = dense_gemm(DType::F32, OutType::Same, src, rinv_t, n, r, r, dst, "fit_qr", part, s);
        if (e != hipSuccess) return e;
        src = dst;
    }
    return hipSuccess;
}

// Subspace iteration of one side: gram [n][n] float32, omega [n][r]; the result in q.
hipError_t fit_side(const float* gram, const float* omega, int n, int r, int iters, const FitWs& w, void* ws,
                    int32_t* status, bool& reset, hipStream_t s) {
    float* q = at<float>(ws, w.q);
    float* y = at<float>(ws, w.y);
    float* q1 = at<float>(ws, w.q1);
    float* qt = at<float>(ws, w.qt);
    hipError_t e = orthonormalise(const_cast<float*>(omega), n, r, q1, q, w, ws, status, reset, s);
    for (int it = 0; it < iters && e == hipSuccess; ++it) {
        e = launch_transpose(DType::F32, q, n, r, qt, s);  // Q^T [r][n]: the GEMM's weight rows
        if (e == hipSuccess) e = dense_gemm(DType::F32, OutType::Same, gram, qt, n, n, r, y, "fit_power", at<float>(ws, w.gpart), s);
        if (e == hipSuccess) e = orthonormalise(y, n, r, q1, q, w, ws, status, reset, s);
    }
    return e;
}

}  // namespace

ec2moe_status ec2moe_lowrank_fit_workspace_size(const ec2moe_codec_desc* desc, size_t* bytes) {
    if (ec2moe_status st = check_codec_desc(desc); st != EC2MOE_OK) return st;
    REQUIRE_PTR(bytes);
    *bytes = fit_ws(desc).total;
    return ok();
}

ec2moe_status ec2moe_lowrank_fit(const ec2moe_codec_desc* desc, const void* x, const float* omega_u,
                                 const float* omega_v, int32_t iters, void* u, void* v, int32_t* status,
                                 void* ws, size_t ws_bytes, hipStream_t stream) {
    if (ec2moe_status st = check_codec_desc(desc); st != EC2MOE_OK) return st;
    const FitWs w = fit_ws(desc);
    if (ec2moe_status st = check_ws(ws, ws_bytes, w.total); st != EC2MOE_OK) return st;
    REQUIRE(desc->n_slices >= 1 && desc->h >= 1, EC2MOE_ERR_INVALID_ARGUMENT, "fitting needs at least one slice of one row");
    REQUIRE(iters >= 0 && iters <= 64, EC2MOE_ERR_INVALID_ARGUMENT, "iters %d outside [0, 64]", iters);
    REQUIRE(static_cast<int64_t>(desc->n_slices) * desc->h % 8 == 0, EC2MOE_ERR_UNSUPPORTED,
            "c*h = %lld is not a multiple of 8", static_cast<long long>(desc->n_slices) * desc->h);
    REQUIRE(static_cast<int64_t>(desc->n_slices) * desc->h * desc->w * elem_bytes(static_cast<DType>(desc->dtype)) <
                (int64_t(1) << 32), EC2MOE_ERR_UNSUPPORTED, "calibration block too large for 32-bit byte offsets");
    REQUIRE_PTR(x); REQUIRE_PTR(omega_u); REQUIRE_PTR(omega_v); REQUIRE_PTR(u); REQUIRE_PTR(v);
    REQUIRE_ALIGNED(x); REQUIRE_ALIGNED(omega_u); REQUIRE_ALIGNED(omega_v); REQUIRE_ALIGNED(u); REQUIRE_ALIGNED(v);
    const DType dt = static_cast<DType>(desc->dtype);
    const int c = desc->n_slices, h = desc->h, wd = desc->w;
    float* gram = at<float>(ws, w.gram);
    void* xt = at<void>(ws, w.xt);
    float* part = at<float>(ws, w.gpart);
    bool reset = true;
    // A = sum_s X_s X_s^T [h][h]: the mode-1 unfolding times itself (K = c*w)
    const void* xu = x;
    hipError_t e = hipSuccess;
    if (c > 1) {
        e = launch_unfold(dt, x, c, h, wd, xt, stream);
        xu = xt;
    }
    if (e == hipSuccess) e = dense_gemm(dt, OutType::F32, xu, xu, h, c * wd, h, gram, "fit_gram_a", part, stream);
    if (e == hipSuccess) e = fit_side(gram, omega_u, h, desc->r_h, iters, w, ws, status, reset, stream);
    if (e == hipSuccess) {
        const int64_t nu = static_cast<int64_t>(h) * desc->r_h;
        e = dt == DType::BF16 ? launch_f32_to_bf16(at<float>(ws, w.q), nu, u, stream)
                              : hipMemcpyAsync(u, at<float>(ws, w.q), nu * 4, hipMemcpyDeviceToDevice, stream);
    }
    // B = sum_s X_s^T X_s [w][w]: X^T [w][c*h] times itself (K = c*h)
    if (e == hipSuccess) e = launch_transpose(dt, x, c * h, wd, xt, stream);
    if (e == hipSuccess) e = dense_gemm(dt, OutType::F32, xt, xt, wd, c * h, wd, gram, "fit_gram_b", part, stream);
    if (e == hipSuccess) e = fit_side(gram, omega_v, wd, desc->r_w, iters, w, ws, status, reset, stream);
    if (e == hipSuccess) {
        const int64_t nv = static_cast<int64_t>(wd) * desc->r_w;
        e = dt == DType::BF16 ? launch_f32_to_bf16(at<float>(ws, w.q), nv, v, stream)
                              : hipMemcpyAsync(v, at<float>(ws, w.q), nv * 4, hipMemcpyDeviceToDevice, stream);
    }
    return hip_status(e, "lowrank_fit launch");
}

ec2moe_status ec2moe_profile_enable(int32_t enable) {
    Profiler& p = prof();
    std::lock_guard<std::mutex> lk(p.mu);
    p.enabled = enable != 0;
    return ok();
}

ec2moe_status ec2moe_profile_select(const char* name) {
    Profiler& p = prof();
    std::lock_guard<std::mutex> lk(p.mu);
    p.only = name ? name : "";
    return ok();
}

ec2moe_status ec2moe_profile_collect(ec2moe_kernel_stat* out, int32_t max_entries, int32_t* n_out) {
    REQUIRE_PTR(n_out);
    REQUIRE(max_entries >= 0, EC2MOE_ERR_INVALID_ARGUMENT, "max_entries < 0");
    REQUIRE(max_entries == 0 || out != nullptr, EC2MOE_ERR_INVALID_ARGUMENT, "out is NULL");
    Profiler& p = prof();
    std::lock_guard<std::mutex> lk(p.mu);
    std::vector<int64_t> launches(p.names.size(), 0);
    std::vector<double> ms(p.names.size(), 0.0);
    hipError_t err = hipSuccess;
    for (const ProfRecord& r : p.records) {
        if (err == hipSuccess) err = hipEventSynchronize(r.stop);
        float t = 0.f;
        if (err == hipSuccess) err = hipEventElapsedTime(&t, r.start, r.stop);
        launches[r.name_id] += 1;
        ms[r.name_id] += t;
        p.pool.push_back(r.start);
        p.pool.push_back(r.stop);
    }
    p.records.clear();
    int n = 0;
    for (size_t i = 0; i < p.names.size(); ++i) {
        if (launches[i] == 0) continue;
        if (n < max_entries) {
            std::memset(out[n].name, 0, sizeof out[n].name);
            std::strncpy(out[n].name, p.names[i].c_str(), sizeof out[n].name - 1);
            out[n].launches = launches[i];
            out[n].total_ms = ms[i];
        }
        ++n;
    }
    *n_out = std::min(n, max_entries);
    return hip_status(err, "profile collect");
}

}  // extern "C"
