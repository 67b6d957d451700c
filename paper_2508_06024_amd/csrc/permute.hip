// Dispatch of (token, slot) assignments to per-expert segments, for gfx950.
//
// The assignments a = t*k + j are sorted stably by expert id with integer work only:
//   1. count:   each 1024-assignment chunk builds an LDS histogram over the experts;
//   2. scan:    one workgroup turns the chunk counts into segment offsets and the
//               first position of every (chunk, expert) pair;
//   3. scatter: each wave walks 256 consecutive assignments 64 at a time; lanes with
//               the same expert find each other with one ballot per bit of the expert
//               id, so the rank inside the 64 comes from a popcount and the order of
//               the input is kept.
// Up to 65536 assignments the three steps run in one launch (perm_onepass_kernel), with
// the counts of step 1 recomputed by every workgroup instead of exchanged through memory.
// No floating point and no global atomics: the result is unique and deterministic.
#include "device_common.h"
#include "internal.h"

#include <algorithm>
#include <mutex>

namespace ec2moe {

// Per-chunk expert counts of the chunked path for callers that cannot allocate: one array
// per GPU, held until the process ends. Host code never uses this name as an address (on
// the host it only stands for the symbol): permute_static_counts() looks up each device's
// copy with hipGetSymbolAddress and the kernels receive that pointer.
static __device__ __align__(256) int32_t scratch[kPermStaticCountWords];

namespace {

constexpr int kWaveItems = kPermChunk / 4;  // assignments per wave per chunk
static_assert(kWaveItems % 64 == 0, "chunk must split into whole wave passes");

__global__ __launch_bounds__(256) void perm_count_kernel(const int32_t* __restrict__ idx, int64_t n,
                                                         int M, int32_t* __restrict__ counts) {
    __shared__ int hist[256];
    for (int e = threadIdx.x; e < M; e += 256) hist[e] = 0;
    __syncthreads();
    const int64_t base = static_cast<int64_t>(blockIdx.x) * kPermChunk;
    for (int i = threadIdx.x; i < kPermChunk; i += 256) {
        const int64_t a = base + i;
        if (a < n) {
            const int e = idx[a];
            if (e >= 0 && e < M) atomicAdd(&hist[e], 1);
        }
    }
    __syncthreads();
    for (int e = threadIdx.x; e < M; e += 256) counts[static_cast<int64_t>(blockIdx.x) * M + e] = hist[e];
}

// counts[c][e] -> absolute first position of chunk c's assignments to expert e. Each expert's
// column is walked 8 chunks at a time (loads in flight together); the expert totals are
// scanned by one wave (lane l owns experts 4 l .. 4 l + 3).
__global__ __launch_bounds__(256) void perm_scan_kernel(int32_t* __restrict__ counts, int n_chunks, int M,
                                                        int32_t* __restrict__ seg) {
    __shared__ int total[256];
    const int e = threadIdx.x;
    const int lane = threadIdx.x & 63;
    int run = 0;
    if (e < M) {
        for (int c0 = 0; c0 < n_chunks; c0 += 8) {
            int v[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) v[j] = c0 + j < n_chunks ? counts[static_cast<int64_t>(c0 + j) * M + e] : 0;
#pragma unroll
            for (int j = 0; j < 8; ++j)
                if (c0 + j < n_chunks) {
                    counts[static_cast<int64_t>(c0 + j) * M + e] = run;
                    run += v[j];
                }
        }
        total[e] = run;
    }
    __syncthreads();
    if (threadIdx.x < 64) {
        int v[4], sum = 0;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int x = 4 * lane + q;
            v[q] = x < M ? total[x] : 0;
            sum += v[q];
        }
        int inc = sum;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const int t = __shfl_up(inc, off);
            if (lane >= off) inc += t;
        }
        int r = inc - sum;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int x = 4 * lane + q;
            if (x < M) total[x] = r;
            r += v[q];
        }
        if (lane == 63) seg[M] = inc;
    }
    __syncthreads();
    if (e < M) {
        const int start = total[e];
        seg[e] = start;
        for (int c0 = 0; c0 < n_chunks; c0 += 8) {
            int v[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) v[j] = c0 + j < n_chunks ? counts[static_cast<int64_t>(c0 + j) * M + e] : 0;
#pragma unroll
            for (int j = 0; j < 8; ++j)
                if (c0 + j < n_chunks) counts[static_cast<int64_t>(c0 + j) * M + e] = v[j] + start;
        }
    }
}

__global__ __launch_bounds__(256) void perm_scatter_kernel(const int32_t* __restrict__ idx, int64_t n, int top_k,
                                                           int M, const int32_t* __restrict__ chunk_base,
                                                           int32_t* __restrict__ perm_src,
                                                           int32_t* __restrict__ inv_perm) {
    __shared__ int wcount[4][256];
    __shared__ int wpos[4][256];
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    for (int i = threadIdx.x; i < 4 * 256; i += 256) (&wcount[0][0])[i] = 0;
    __syncthreads();
    const int64_t wbeg = static_cast<int64_t>(blockIdx.x) * kPermChunk + static_cast<int64_t>(wave) * kWaveItems;
    for (int i = lane; i < kWaveItems; i += 64) {
        const int64_t a = wbeg + i;
        if (a < n) {
            const int e = idx[a];
            if (e >= 0 && e < M) atomicAdd(&wcount[wave][e], 1);
        }
    }
    __syncthreads();
    for (int e = threadIdx.x; e < M; e += 256) {
        int b = chunk_base[static_cast<int64_t>(blockIdx.x) * M + e];
        for (int w = 0; w < 4; ++w) {
            wpos[w][e] = b;
            b += wcount[w][e];
        }
    }
    __syncthreads();

    int nbits = 0;
    while ((1 << nbits) < M) ++nbits;
    const uint64_t lt_mask = (1ull << lane) - 1ull;
    for (int s = 0; s < kWaveItems; s += 64) {
        const int64_t a = wbeg + s + lane;
        int e = -1;
        if (a < n) {
            e = idx[a];
            if (e < 0 || e >= M) {
                inv_perm[a] = -1;
                e = -1;
            }
        }
        const bool valid = e >= 0;
        uint64_t peers = __ballot(valid);
        for (int b = 0; b < nbits; ++b) {
            const bool bit = valid && ((e >> b) & 1);
            const uint64_t ones = __ballot(bit);
            peers &= bit ? ones : ~ones;
        }
        if (valid) {
            const int rank = __popcll(peers & lt_mask);
            const int pos = wpos[wave][e] + rank;
            perm_src[pos] = static_cast<int32_t>(a / top_k);
            inv_perm[a] = pos;
        }
        // every lane has read its base; the first lane of each expert advances it
        __builtin_amdgcn_wave_barrier();
        if (valid && (peers & lt_mask) == 0) wpos[wave][e] += __popcll(peers);
        __builtin_amdgcn_wave_barrier();
    }
}

// Up to kOnePassMax assignments the three steps take one launch and need no workspace: a
// workgroup per chunk of kPermChunk assignments, each counting the whole index array (a few
// tens of KB, read from L2) split into the assignments before its chunk, in it (per wave)
// and after it. That gives every segment's offset and the position of the chunk inside each
// segment without any exchange between workgroups; wave w then scatters the w-th run of 64
// assignments of the chunk with ballot ranks, which keep the input order.
constexpr int kOneWaves = kPermChunk / 64;  // one 64-assignment run per wave
constexpr int64_t kOnePassMax = 65536;      // the redundant counting reads n^2 / 1024 indices in all

__global__ __launch_bounds__(64 * kOneWaves) void perm_onepass_kernel(const int32_t* __restrict__ idx, int64_t n,
                                                                      int top_k, int M, int32_t* __restrict__ seg,
                                                                      int32_t* __restrict__ perm_src,
                                                                      int32_t* __restrict__ inv_perm) {
    constexpr int NT = 64 * kOneWaves;
    __shared__ int before[256];              // assignments to each expert before this chunk
    __shared__ int after[256];               // ... after it
    __shared__ int start[256];               // expert totals, then segment offsets
    __shared__ int wpos[kOneWaves][256];     // this chunk's counts per (wave, expert), then positions
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    for (int i = threadIdx.x; i < 256; i += NT) {
        before[i] = 0;
        after[i] = 0;
    }
    for (int i = threadIdx.x; i < kOneWaves * 256; i += NT) (&wpos[0][0])[i] = 0;
    __syncthreads();
    const int64_t cbeg = static_cast<int64_t>(blockIdx.x) * kPermChunk;
    const int64_t cend = std::min<int64_t>(n, cbeg + kPermChunk);
    const int64_t a_mine = cbeg + 64 * wave + lane;
    const int e_mine = a_mine < cend ? idx[a_mine] : -1;
    const bool valid = e_mine >= 0 && e_mine < M;
    // everything outside the chunk, U loads in flight per thread
    constexpr int U = 16;
    for (int64_t s0 = 0; s0 < n; s0 += static_cast<int64_t>(NT) * U) {
        int ev[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t a = s0 + static_cast<int64_t>(NT) * u + threadIdx.x;
            ev[u] = (a < n && (a < cbeg || a >= cend)) ? idx[a] : -1;
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t a = s0 + static_cast<int64_t>(NT) * u + threadIdx.x;
            if (ev[u] >= 0 && ev[u] < M) atomicAdd(a < cbeg ? &before[ev[u]] : &after[ev[u]], 1);
        }
    }
    if (valid) atomicAdd(&wpos[wave][e_mine], 1);
    __syncthreads();
    // per expert: the waves' runs inside the chunk, and the expert's total
    if (threadIdx.x < M) {
        const int e = threadIdx.x;
        int run = 0;
#pragma unroll
        for (int w = 0; w < kOneWaves; ++w) {
            const int c = wpos[w][e];
            wpos[w][e] = run;
            run += c;
        }
        start[e] = before[e] + run + after[e];
    }
    __syncthreads();
    // exclusive scan of the totals over experts: lane l of wave 0 owns experts 4 l .. 4 l + 3
    if (wave == 0) {
        int v[4], sum = 0;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int e = 4 * lane + q;
            v[q] = e < M ? start[e] : 0;
            sum += v[q];
        }
        int inc = sum;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const int t = __shfl_up(inc, off);
            if (lane >= off) inc += t;
        }
        int run = inc - sum;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int e = 4 * lane + q;
            if (e < M) {
                start[e] = run;
                if (blockIdx.x == 0) seg[e] = run;
            }
            run += v[q];
        }
        if (blockIdx.x == 0 && lane == 63) seg[M] = inc;
    }
    __syncthreads();
    if (threadIdx.x < M) {
        const int e = threadIdx.x;
        const int base = start[e] + before[e];
#pragma unroll
        for (int w = 0; w < kOneWaves; ++w) wpos[w][e] += base;
    }
    __syncthreads();
    if (a_mine >= cend) return;  // the wave's run ends inside the chunk: the ballots below skip these lanes
    int nbits = 0;
    while ((1 << nbits) < M) ++nbits;
    const uint64_t lt_mask = (1ull << lane) - 1ull;
    uint64_t peers = __ballot(valid);
    for (int b = 0; b < nbits; ++b) {
        const bool bit = valid && ((e_mine >> b) & 1);
        const uint64_t ones = __ballot(bit);
        peers &= bit ? ones : ~ones;
    }
    if (valid) {
        const int pos = wpos[wave][e_mine] + __popcll(peers & lt_mask);
        perm_src[pos] = static_cast<int32_t>(a_mine / top_k);
        inv_perm[a_mine] = pos;
    } else {
        inv_perm[a_mine] = -1;
    }
}

// Rows past the valid segments (only when some expert ids were out of range) and
// source ids outside [0, n_src) are written as zeros.
__global__ __launch_bounds__(256) void gather_rows_kernel(const char* __restrict__ x,
                                                          const int32_t* __restrict__ perm_src,
                                                          const int32_t* __restrict__ seg_end, int64_t n_src,
                                                          int64_t rows, int row_chunks, char* __restrict__ out) {
    const int64_t total = rows * row_chunks;
    const int64_t valid_rows = *seg_end;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; i < total;
         i += static_cast<int64_t>(gridDim.x) * 256) {
        const int64_t r = i / row_chunks;
        const int c = static_cast<int>(i - r * row_chunks);
        const int64_t src = r < valid_rows ? perm_src[r] : -1;
        const uint4 v = (src >= 0 && src < n_src) ? ldg16(x + (src * row_chunks + c) * 16) : make_uint4(0, 0, 0, 0);
        stg16(out + (r * row_chunks + c) * 16, v);
    }
}

}  // namespace

hipError_t launch_permute(const int32_t* topk_idx, int64_t n_assign, int top_k, int n_experts,
                          int32_t* chunk_counts, int32_t* seg_offsets, int32_t* perm_src,
                          int32_t* inv_perm, hipStream_t s) {
    if (n_assign <= kOnePassMax) {
        ProfileScope prof("perm_onepass", s);
        const int grid = std::max(1, perm_chunks(n_assign));
        hipLaunchKernelGGL(perm_onepass_kernel, dim3(grid), dim3(64 * kOneWaves), 0, s, topk_idx, n_assign, top_k,
                           n_experts, seg_offsets, perm_src, inv_perm);
        return hipGetLastError();
    }
    const int chunks = perm_chunks(n_assign);
    if (chunks == 0) {
        ProfileScope prof("perm_scan", s);
        hipLaunchKernelGGL(perm_scan_kernel, dim3(1), dim3(256), 0, s, chunk_counts, 0, n_experts, seg_offsets);
        return hipGetLastError();
    }
    {
        ProfileScope prof("perm_count", s);
        hipLaunchKernelGGL(perm_count_kernel, dim3(chunks), dim3(256), 0, s, topk_idx, n_assign, n_experts,
                           chunk_counts);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    {
        ProfileScope prof("perm_scan", s);
        hipLaunchKernelGGL(perm_scan_kernel, dim3(1), dim3(256), 0, s, chunk_counts, chunks, n_experts,
                           seg_offsets);
    }
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    {
        ProfileScope prof("perm_scatter", s);
        hipLaunchKernelGGL(perm_scatter_kernel, dim3(chunks), dim3(256), 0, s, topk_idx, n_assign, top_k,
                           n_experts, chunk_counts, perm_src, inv_perm);
    }
    return hipGetLastError();
}

hipError_t permute_static_counts(int32_t** counts) {
    constexpr int kMaxDevices = 64;
    static std::mutex mu;
    static int32_t* addr[kMaxDevices] = {};
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lk(mu);
    if (addr[dev] == nullptr) {
        void* p = nullptr;
        // once per device, with that device current: its own copy of the array
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        addr[dev] = static_cast<int32_t*>(p);
    }
    *counts = addr[dev];
    return hipSuccess;
}

hipError_t launch_gather_rows(DType dt, const void* x, int64_t n_src, const int32_t* perm_src,
                              const int32_t* seg_end, int64_t n_rows, int d, void* x_perm, hipStream_t s) {
    if (n_rows == 0) return hipSuccess;
    const int row_chunks = static_cast<int>(d * elem_bytes(dt) / 16);
    const int64_t total = n_rows * row_chunks;
    const int grid = static_cast<int>(std::min<int64_t>((total + 255) / 256, 8192));
    ProfileScope prof("gather_rows", s);
    hipLaunchKernelGGL(gather_rows_kernel, dim3(grid), dim3(256), 0, s, static_cast<const char*>(x), perm_src,
                       seg_end, n_src, n_rows, row_chunks, static_cast<char*>(x_perm));
    return hipGetLastError();
}

}  // namespace ec2moe
