// GlobalRandK sparsification (Sec. 3.3-3.4) for gfx950: a uniformly random
// K-subset of the d coordinates, shared by every worker, then gather and
// scatter between the full vectors and the dense [M][K] sub-problem that the
// quantiser kernels handle unchanged.
//
// Selection.  Coordinate i has the 64-bit key (hi, lo): hi is word i%4 of
// Philox block (i/4, 0, purpose 2), lo the same word of block (i/4, 0,
// purpose 3).  The K coordinates with the smallest (hi, lo, i) are chosen.
// Keys are regenerated in every pass (no key array in memory):
//   1. per-block LDS histograms of hi >> 20 (4096 bins), merged with atomics;
//   2. one block finds the bin b1 holding the K-th key and how many keys of
//      it are still needed;
//   3. keys in bin b1 histogram (hi >> 8) & 0xFFF (sparse global atomics);
//   4. one block finds the sub-bin b2;
//   5. keys whose top 24 bits are (b1, b2) are collected with their low
//      words (expected d / 2^24 of them, at most kRandkCandidates);
//   6. one block ranks the candidates and takes the (key, index) threshold;
//   7. the coordinates at or below the threshold (exactly K) are written in
//      increasing order: contiguous per-block ranges are counted, the counts
//      scanned, and each block then writes its selections at its offset,
//      ordered inside the block by wave ballots.
#include <stdint.h>

#include "uq_device.hpp"
#include "uq_launch.hpp"

namespace uq {

constexpr int kRkBins = 4096;
constexpr int kRkSortThreads = 1024;

struct RandkControl {
    uint32_t b1, need1, b2, need2;  // bins found by the two scans
    uint32_t n_cand, n_sel;         // append counters
    uint32_t thr_hi, thr_lo, thr_idx;
    uint32_t pad[7];
};

constexpr int kRkMaxBlocks = 2048;  // ordered-compaction blocks

struct RandkWorkspace {
    uint32_t hist1[kRkBins];
    uint32_t hist2[kRkBins];
    RandkControl ctl;
    uint32_t cand[kRandkCandidates][3];  // (hi, lo, index)
    uint32_t block_count[kRkMaxBlocks];
    uint32_t block_offset[kRkMaxBlocks];
};

__device__ __forceinline__ uint4 selection_block(uint32_t q, uint32_t purpose, uint32_t key0, uint32_t key1)
{
    return philox4x32_10(q, 0u, 0u, purpose, key0, key1);
}

__device__ __forceinline__ uint32_t word_of(uint4 w, int j)
{
    return j == 0 ? w.x : (j == 1 ? w.y : (j == 2 ? w.z : w.w));
}

__global__ __launch_bounds__(kBlock) void k_rk_init(RandkWorkspace* __restrict__ ws)
{
    for (int b = threadIdx.x; b < kRkBins; b += kBlock) {
        ws->hist1[b] = 0u;
        ws->hist2[b] = 0u;
    }
    if (threadIdx.x < sizeof(RandkControl) / 4)
        reinterpret_cast<uint32_t*>(&ws->ctl)[threadIdx.x] = 0u;
}

// Pass 1: histogram of the top 12 bits of hi.
__global__ __launch_bounds__(kBlock) void k_rk_hist1(int64_t d, uint32_t key0, uint32_t key1,
                                                     RandkWorkspace* __restrict__ ws)
{
    __shared__ uint32_t h[kRkBins];
    for (int b = threadIdx.x; b < kRkBins; b += kBlock)
        h[b] = 0u;
    __syncthreads();
    const int64_t nq = (d + 3) >> 2;
    for (int64_t q = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; q < nq;
         q += static_cast<int64_t>(gridDim.x) * kBlock) {
        const uint4 w = selection_block(static_cast<uint32_t>(q), 2u, key0, key1);
#pragma unroll
        for (int j = 0; j < 4; ++j)
            if ((q << 2) + j < d)
                atomicAdd(&h[word_of(w, j) >> 20], 1u);
    }
    __syncthreads();
    for (int b = threadIdx.x; b < kRkBins; b += kBlock)
        if (h[b] != 0u)
            atomicAdd(&ws->hist1[b], h[b]);
}

// Scans (one block): the bin whose cumulative count first reaches `need`.
__global__ __launch_bounds__(kBlock) void k_rk_scan(RandkWorkspace* __restrict__ ws, int level, uint32_t K)
{
    __shared__ uint32_t part[kBlock];
    const uint32_t* hist = level == 1 ? ws->hist1 : ws->hist2;
    const uint32_t need = level == 1 ? K : ws->ctl.need1;
    constexpr int per = kRkBins / kBlock;  // 16 bins per thread
    uint32_t local = 0u;
#pragma unroll
    for (int j = 0; j < per; ++j)
        local += hist[threadIdx.x * per + j];
    part[threadIdx.x] = local;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t cum = 0u;
        int t = 0;
        while (t < kBlock - 1 && cum + part[t] < need)
            cum += part[t++];
        int b = t * per;
        while (b < kRkBins - 1 && cum + hist[b] < need)
            cum += hist[b++];
        if (level == 1) {
            ws->ctl.b1 = static_cast<uint32_t>(b);
            ws->ctl.need1 = need - cum;
        } else {
            ws->ctl.b2 = static_cast<uint32_t>(b);
            ws->ctl.need2 = need - cum;
        }
    }
}

// Pass 2: keys in bin b1 histogram bits 19..8 of hi.
__global__ __launch_bounds__(kBlock) void k_rk_hist2(int64_t d, uint32_t key0, uint32_t key1,
                                                     RandkWorkspace* __restrict__ ws)
{
    const uint32_t b1 = ws->ctl.b1;
    const int64_t nq = (d + 3) >> 2;
    for (int64_t q = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; q < nq;
         q += static_cast<int64_t>(gridDim.x) * kBlock) {
        const uint4 w = selection_block(static_cast<uint32_t>(q), 2u, key0, key1);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const uint32_t hi = word_of(w, j);
            if ((q << 2) + j < d && (hi >> 20) == b1)
                atomicAdd(&ws->hist2[(hi >> 8) & 0xFFFu], 1u);
        }
    }
}

// Pass 3: collect the keys whose top 24 bits are (b1, b2), with low words.
__global__ __launch_bounds__(kBlock) void k_rk_collect(int64_t d, uint32_t key0, uint32_t key1,
                                                       RandkWorkspace* __restrict__ ws)
{
    const uint32_t prefix = (ws->ctl.b1 << 12) | ws->ctl.b2;
    const int64_t nq = (d + 3) >> 2;
    for (int64_t q = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; q < nq;
         q += static_cast<int64_t>(gridDim.x) * kBlock) {
        const uint4 w = selection_block(static_cast<uint32_t>(q), 2u, key0, key1);
        bool any = false;
#pragma unroll
        for (int j = 0; j < 4; ++j)
            any = any || (((q << 2) + j < d) && (word_of(w, j) >> 8) == prefix);
        if (any) {
            const uint4 l = selection_block(static_cast<uint32_t>(q), 3u, key0, key1);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int64_t i = (q << 2) + j;
                if (i < d && (word_of(w, j) >> 8) == prefix) {
                    const uint32_t slot = atomicAdd(&ws->ctl.n_cand, 1u);
                    if (slot < static_cast<uint32_t>(kRandkCandidates)) {
                        ws->cand[slot][0] = word_of(w, j);
                        ws->cand[slot][1] = word_of(l, j);
                        ws->cand[slot][2] = static_cast<uint32_t>(i);
                    }
                }
            }
        }
    }
}

__device__ __forceinline__ bool key_less(uint32_t ah, uint32_t al, uint32_t ai, uint32_t bh, uint32_t bl,
                                         uint32_t bi)
{
    return ah != bh ? ah < bh : (al != bl ? al < bl : ai < bi);
}

// One block: the candidate whose rank among the candidates (by hi, lo,
// index; all distinct) is need2 - 1 is the threshold.  About d / 2^24
// candidates are expected, so a direct count of smaller keys is cheapest.
__global__ __launch_bounds__(kRkSortThreads) void k_rk_threshold(RandkWorkspace* __restrict__ ws)
{
    const uint32_t n = min(ws->ctl.n_cand, static_cast<uint32_t>(kRandkCandidates));
    const uint32_t want = ws->ctl.need2 - 1u;
    for (uint32_t t = threadIdx.x; t < n; t += kRkSortThreads) {
        const uint32_t h = ws->cand[t][0], l = ws->cand[t][1], i = ws->cand[t][2];
        uint32_t rank = 0u;
        for (uint32_t u = 0; u < n; ++u)
            rank += key_less(ws->cand[u][0], ws->cand[u][1], ws->cand[u][2], h, l, i) ? 1u : 0u;
        if (rank == want) {
            ws->ctl.thr_hi = h;
            ws->ctl.thr_lo = l;
            ws->ctl.thr_idx = i;
        }
    }
}

// Whether coordinate i = 4q + j (j < 4) is at or below the threshold.
__device__ __forceinline__ uint32_t selected_mask(int64_t q, int64_t d, uint32_t key0, uint32_t key1, uint32_t th,
                                                  uint32_t tl, uint32_t ti)
{
    const uint4 w = selection_block(static_cast<uint32_t>(q), 2u, key0, key1);
    bool tie = false;
#pragma unroll
    for (int j = 0; j < 4; ++j)
        tie = tie || (((q << 2) + j < d) && word_of(w, j) == th);
    uint4 l = make_uint4(0u, 0u, 0u, 0u);
    if (tie)
        l = selection_block(static_cast<uint32_t>(q), 3u, key0, key1);
    uint32_t mask = 0u;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int64_t i = (q << 2) + j;
        const uint32_t hi = word_of(w, j);
        const bool take = i < d && (hi < th || (hi == th && !key_less(th, tl, ti, hi, word_of(l, j),
                                                                       static_cast<uint32_t>(i))));
        mask |= take ? (1u << j) : 0u;
    }
    return mask;
}

// Block b owns coordinates [b * chunk, (b + 1) * chunk): pass 4 counts its
// selections, pass 5 writes them in order at the scanned offset.
__global__ __launch_bounds__(kBlock) void k_rk_count(int64_t d, int64_t chunk, uint32_t key0, uint32_t key1,
                                                     RandkWorkspace* __restrict__ ws)
{
    __shared__ uint32_t wave_count[kBlock / 64];
    const uint32_t th = ws->ctl.thr_hi, tl = ws->ctl.thr_lo, ti = ws->ctl.thr_idx;
    const int64_t q0 = (static_cast<int64_t>(blockIdx.x) * chunk) >> 2;
    const int64_t q1 = min((static_cast<int64_t>(blockIdx.x) + 1) * chunk, d + 3) >> 2;
    uint32_t count = 0u;
    for (int64_t q = q0 + threadIdx.x; q < q1; q += kBlock)
        count += __builtin_popcount(selected_mask(q, d, key0, key1, th, tl, ti));
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1)
        count += __shfl_xor(count, off, 64);
    if ((threadIdx.x & 63) == 0)
        wave_count[threadIdx.x >> 6] = count;
    __syncthreads();
    if (threadIdx.x == 0)
        ws->block_count[blockIdx.x] = wave_count[0] + wave_count[1] + wave_count[2] + wave_count[3];
}

// One block: exclusive scan of the per-block counts.
__global__ __launch_bounds__(kBlock) void k_rk_offsets(RandkWorkspace* __restrict__ ws, int32_t nblocks)
{
    __shared__ uint32_t part[kBlock];
    const int per = (nblocks + kBlock - 1) / kBlock;
    const int b0 = threadIdx.x * per;
    uint32_t local = 0u;
    for (int b = b0; b < b0 + per && b < nblocks; ++b)
        local += ws->block_count[b];
    part[threadIdx.x] = local;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t run = 0u;
        for (int t = 0; t < kBlock; ++t) {
            const uint32_t x = part[t];
            part[t] = run;
            run += x;
        }
    }
    __syncthreads();
    uint32_t run = part[threadIdx.x];
    for (int b = b0; b < b0 + per && b < nblocks; ++b) {
        const uint32_t x = ws->block_count[b];
        ws->block_offset[b] = run;
        run += x;
    }
}

__global__ __launch_bounds__(kBlock) void k_rk_write(int64_t d, int64_t chunk, uint32_t key0, uint32_t key1,
                                                     const RandkWorkspace* __restrict__ ws, uint32_t* __restrict__ sel,
                                                     uint32_t K)
{
    __shared__ uint32_t wave_count[kBlock / 64];
    const uint32_t th = ws->ctl.thr_hi, tl = ws->ctl.thr_lo, ti = ws->ctl.thr_idx;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const uint64_t below = (uint64_t(1) << lane) - 1u;
    uint32_t base = ws->block_offset[blockIdx.x];
    const int64_t q0 = (static_cast<int64_t>(blockIdx.x) * chunk) >> 2;
    const int64_t q1 = min((static_cast<int64_t>(blockIdx.x) + 1) * chunk, d + 3) >> 2;
    // sub-ranges of 1024 coordinates in order: thread t holds group qb + t
    for (int64_t qb = q0; qb < q1; qb += kBlock) {
        const int64_t q = qb + threadIdx.x;
        const uint32_t mask = q < q1 ? selected_mask(q, d, key0, key1, th, tl, ti) : 0u;
        // selections of the lanes before this one in the wave, and the wave's total
        uint32_t before = 0u, total = 0u;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const uint64_t b = __ballot((mask >> j) & 1u);
            before += __popcll(b & below);
            total += __popcll(b);
        }
        if (lane == 0)
            wave_count[wave] = total;
        __syncthreads();
        uint32_t pos = base + before;
        for (int v = 0; v < wave; ++v)
            pos += wave_count[v];
#pragma unroll
        for (int j = 0; j < 4; ++j)
            if ((mask >> j) & 1u) {
                if (pos < K)  // exactly K by construction; the guard keeps writes in bounds
                    sel[pos] = static_cast<uint32_t>((q << 2) + j);
                ++pos;
            }
        base += wave_count[0] + wave_count[1] + wave_count[2] + wave_count[3];
        __syncthreads();  // wave_count is rewritten for the next sub-range
    }
}

// sub[m][j] = g[m][sel[j]]
// (an index >= d reads as 0)
__global__ __launch_bounds__(kBlock) void k_gather(const float* __restrict__ g, int64_t d, int64_t ldg,
                                                   const uint32_t* __restrict__ sel, int64_t K,
                                                   float* __restrict__ sub, int64_t lds)
{
    const int32_t m = blockIdx.y;
    for (int64_t j = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; j < K;
         j += static_cast<int64_t>(gridDim.x) * kBlock) {
        const uint32_t i = sel[j];
        sub[static_cast<int64_t>(m) * lds + j] = i < d ? g[static_cast<int64_t>(m) * ldg + i] : 0.0f;
    }
}

__global__ __launch_bounds__(kBlock) void k_zero(float* __restrict__ out, int64_t d)
{
    const int64_t n4 = d >> 2;
    const f32x4 z = {0.0f, 0.0f, 0.0f, 0.0f};
    for (int64_t q = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; q < n4;
         q += static_cast<int64_t>(gridDim.x) * kBlock)
        store_nt(out + (q << 2), z);
    const int64_t t = (n4 << 2) + static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
    if (blockIdx.x == 0 && t < d)
        out[t] = 0.0f;
}

// (an index >= d is skipped)
__global__ __launch_bounds__(kBlock) void k_scatter(const float* __restrict__ vals, const uint32_t* __restrict__ sel,
                                                    int64_t K, float* __restrict__ out, int64_t d)
{
    for (int64_t j = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; j < K;
         j += static_cast<int64_t>(gridDim.x) * kBlock) {
        const uint32_t i = sel[j];
        if (i < d)
            out[i] = vals[j];
    }
}

size_t randk_workspace_bytes()
{
    return (sizeof(RandkWorkspace) + 255) / 256 * 256;
}

static unsigned key_grid(int64_t d)
{
    const int64_t groups = (d + 3) >> 2;
    int64_t blocks = (groups + kBlock - 1) / kBlock;
    const int64_t cap = grid_cap();
    blocks = blocks < 1 ? 1 : (blocks > cap ? cap : blocks);
    return static_cast<unsigned>(blocks);
}

hipError_t launch_randk_select(int64_t d, int64_t K, uint64_t seed, uint32_t* sel, void* ws_raw, hipStream_t stream)
{
    RandkWorkspace* ws = static_cast<RandkWorkspace*>(ws_raw);
    const uint32_t key0 = static_cast<uint32_t>(seed);
    const uint32_t key1 = static_cast<uint32_t>(seed >> 32);
    const unsigned gx = key_grid(d);
    hipLaunchKernelGGL(k_rk_init, dim3(1), dim3(kBlock), 0, stream, ws);
    // the first histogram merges 4096 LDS bins per block into global memory:
    // few, long-lived blocks keep those atomics to a few per bin
    int64_t hist_blocks = grid_cap() / 32;  // two blocks per compute unit
    hist_blocks = hist_blocks > static_cast<int64_t>(gx) ? static_cast<int64_t>(gx) : hist_blocks;
    hipLaunchKernelGGL(k_rk_hist1, dim3(static_cast<unsigned>(hist_blocks)), dim3(kBlock), 0, stream, d, key0, key1,
                       ws);
    hipLaunchKernelGGL(k_rk_scan, dim3(1), dim3(kBlock), 0, stream, ws, 1, static_cast<uint32_t>(K));
    hipLaunchKernelGGL(k_rk_hist2, dim3(gx), dim3(kBlock), 0, stream, d, key0, key1, ws);
    hipLaunchKernelGGL(k_rk_scan, dim3(1), dim3(kBlock), 0, stream, ws, 2, static_cast<uint32_t>(K));
    hipLaunchKernelGGL(k_rk_collect, dim3(gx), dim3(kBlock), 0, stream, d, key0, key1, ws);
    hipLaunchKernelGGL(k_rk_threshold, dim3(1), dim3(kRkSortThreads), 0, stream, ws);
    // ordered compaction over contiguous chunks (a multiple of 1024 coordinates)
    const int64_t per_block = 1024;
    int64_t chunk = (d + kRkMaxBlocks - 1) / kRkMaxBlocks;
    chunk = (chunk + per_block - 1) / per_block * per_block;
    const int32_t nblocks = static_cast<int32_t>((d + chunk - 1) / chunk);
    hipLaunchKernelGGL(k_rk_count, dim3(nblocks), dim3(kBlock), 0, stream, d, chunk, key0, key1, ws);
    hipLaunchKernelGGL(k_rk_offsets, dim3(1), dim3(kBlock), 0, stream, ws, nblocks);
    hipLaunchKernelGGL(k_rk_write, dim3(nblocks), dim3(kBlock), 0, stream, d, chunk, key0, key1, ws, sel,
                       static_cast<uint32_t>(K));
    return hipGetLastError();
}

hipError_t launch_gather(const float* g, int64_t d, int32_t M, int64_t ldg, const uint32_t* sel, int64_t K,
                         float* sub, int64_t lds, hipStream_t stream)
{
    int64_t blocks = (K + kBlock - 1) / kBlock;
    blocks = blocks < 1 ? 1 : blocks;
    hipLaunchKernelGGL(k_gather, dim3(static_cast<unsigned>(blocks), static_cast<unsigned>(M)), dim3(kBlock), 0,
                       stream, g, d, ldg, sel, K, sub, lds);
    return hipGetLastError();
}

hipError_t launch_scatter(const float* vals, const uint32_t* sel, int64_t K, float* out, int64_t d,
                          hipStream_t stream)
{
    int64_t zb = ((d + 3) / 4 + kBlock - 1) / kBlock;
    const int64_t cap = grid_cap();
    zb = zb < 1 ? 1 : (zb > cap ? cap : zb);
    hipLaunchKernelGGL(k_zero, dim3(static_cast<unsigned>(zb)), dim3(kBlock), 0, stream, out, d);
    int64_t sb = (K + kBlock - 1) / kBlock;
    sb = sb < 1 ? 1 : sb;
    hipLaunchKernelGGL(k_scatter, dim3(static_cast<unsigned>(sb)), dim3(kBlock), 0, stream, vals, sel, K, out, d);
    return hipGetLastError();
}

}  // namespace uq
