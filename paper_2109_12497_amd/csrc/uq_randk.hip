// GlobalRandK sparsification (Sec. 3.3-3.4) for gfx950: a uniformly random
// K-subset of the d coordinates, shared by every worker, then gather and
// scatter between the full vectors and the dense [M][K] sub-problem that the
// quantiser kernels handle unchanged.
//
// Selection.  Coordinate i has the 64-bit key (hi, lo): hi is word i%4 of
// Philox block (i/4, 0, purpose 2), lo the same word of block (i/4, 0,
// purpose 3).  The K coordinates with the smallest (hi, lo, i) are chosen.
// Keys are regenerated in every pass (no key array in memory).
//
// For K <= kRkSortMax the host first brackets the K-th key: hi is uniform, so
// the count of keys below any x is binomial and an interval [x_lo, x_hi] of hi
// ten standard deviations either side of K holds the K-th key except with
// probability below 1e-20.  One pass over the keys appends every key below
// x_lo to kRkShards staging lists (each wave adds its selections with one
// atomic, spread over the lists' counters: device-scope atomics on one
// address serialise) and collects the ~20 sqrt(K) keys inside the interval
// with their low words; each of the 64 blocks that sort the lists (one slice
// of the index range each) checks that the interval held the K-th key and
// picks the smallest candidates itself.  Should the bracket miss, every such
// block computes the exact selection itself with the steps below, so the
// result never depends on it.
//
// The histogram passes (K > kRkSortMax, or by the test hook):
//   1. per-block LDS histograms of hi >> 24 (256 bins), merged with atomics;
//   2. every block of the next pass finds the bin b1 holding the K-th key
//      (and how many of its keys are still needed) from that histogram, and
//      keys in bin b1 histogram (hi >> 12) & 0xFFF (global atomics);
//   3. one block finds the sub-bin b2;
//   4. keys whose top 20 bits are (b1, b2) are collected with their low
//      words (expected d / 2^20 of them, at most kRandkCandidates), and for
//      K <= kRkSortMax the keys below that prefix are staged as above;
//   5. one block ranks the candidates and takes the (key, index) threshold;
//   6. the coordinates at or below the threshold (exactly K) are output in
//      increasing order: by the sort above, or for larger K contiguous
//      per-block ranges are counted, the counts scanned, and each block
//      writes its selections at its offset, ordered by wave ballots.
// The key passes run persistent grids, four independent Philox blocks per
// thread and iteration.
#include <stddef.h>
#include <stdint.h>

#include <atomic>
#include <cmath>

#include "uq_device.hpp"
#include "uq_launch.hpp"

namespace uq {

constexpr int kRkBins1 = 256;    // level 1: hi >> 24
constexpr int kRkBins2 = 4096;   // level 2: (hi >> 12) & 0xFFF
constexpr int kRkSortThreads = 1024;
constexpr int kRkSortMax = 16384;  // largest K sorted by one block
constexpr int kRkShards = 64;      // staging lists of the K <= kRkSortMax path
constexpr int kRkUnroll = 4;       // Philox blocks per thread and iteration
constexpr int kRkCopies = 16;      // level-1 histogram copies the blocks merge into
constexpr int kRkLine = 64;        // uint32 per 256-byte line: one atomic counter per line
constexpr int kRkShardCand = 256;  // bracket candidates per staging list

struct RandkControl {
    uint32_t b1, need1, b2, need2;  // bins found by the two scans
    uint32_t n_cand, cand_cap;      // candidate append counter; candidates kept (<= kRandkCandidates)
    uint32_t thr_hi, thr_lo, thr_idx;
    uint32_t x_lo, x_hi;            // collection interval of hi (inclusive)
    uint32_t exact;                 // 1: the candidates overflowed, the sort takes the exact path
    uint32_t pad[4];
};

constexpr int kRkMaxBlocks = 2048;  // ordered-compaction blocks

// Device-scope atomics execute at the memory side and serialise per cache
// line, so counters that many waves hit live on lines of their own and the
// level-1 histogram is merged into kRkCopies copies.
struct RandkWorkspace {
    uint32_t hist1[kRkCopies][kRkBins1];
    uint32_t hist2[kRkBins2];
    RandkControl ctl;
    uint32_t cand[kRandkCandidates][3];  // (hi, lo, index)
    uint32_t block_count[kRkMaxBlocks];
    uint32_t block_offset[kRkMaxBlocks];
    uint32_t n_stage[kRkShards][kRkLine];     // staging list lengths (element 0 of each line)
    uint32_t stage[kRkShards][kRkSortMax];    // unordered selections (K <= kRkSortMax)
    uint32_t n_bcand[kRkShards][kRkLine];     // bracket candidates per list (element 0 of each line)
    uint32_t bcand[kRkShards][kRkShardCand][3];  // (hi, lo, index)
};

__device__ __forceinline__ uint4 selection_block(uint32_t q, uint32_t purpose, uint32_t key0, uint32_t key1)
{
    return philox4x32_10(q, 0u, 0u, purpose, key0, key1);
}

__device__ __forceinline__ uint32_t word_of(uint4 w, int j)
{
    return j == 0 ? w.x : (j == 1 ? w.y : (j == 2 ? w.z : w.w));
}

// Inclusive scan of one value per thread over a block of THREADS threads
// (scratch: THREADS / 64 words of LDS).
template <int THREADS = kBlock>
__device__ __forceinline__ uint32_t block_inclusive_scan(uint32_t x, uint32_t* scratch)
{
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const uint32_t y = __shfl_up(x, off, 64);
        if (lane >= off)
            x += y;
    }
    if (lane == 63)
        scratch[wave] = x;
    __syncthreads();
    uint32_t before = 0u;
    for (int v = 0; v < wave; ++v)
        before += scratch[v];
    __syncthreads();  // scratch may be reused by the caller
    return x + before;
}

// The bin of hist[0 .. THREADS * PER) where the cumulative count first
// reaches `need` (1 <= need <= the total), and how many keys of that bin are
// still needed.  Thread t owns bins [t * PER, (t + 1) * PER); the owner of the
// crossing writes *bin and *rest.
template <int PER, int THREADS = kBlock>
__device__ __forceinline__ void find_bin(const uint32_t* hist, uint32_t need, uint32_t* scratch, uint32_t* bin,
                                         uint32_t* rest)
{
    uint32_t v[PER];
    uint32_t s = 0u;
#pragma unroll
    for (int j = 0; j < PER; ++j) {
        v[j] = hist[threadIdx.x * PER + j];
        s += v[j];
    }
    const uint32_t incl = block_inclusive_scan<THREADS>(s, scratch);
    uint32_t cum = incl - s;
    if (cum < need && need <= incl) {
#pragma unroll
        for (int j = 0; j < PER; ++j) {
            if (cum < need && need <= cum + v[j]) {
                *bin = static_cast<uint32_t>(threadIdx.x * PER + j);
                *rest = need - cum;
            }
            cum += v[j];
        }
    }
}

static_assert(kRkCopies * kRkBins1 == kRkBins2, "one zeroing loop covers both histograms");
__global__ __launch_bounds__(kBlock) void k_rk_init(RandkWorkspace* __restrict__ ws, uint32_t x_lo, uint32_t x_hi,
                                                    uint32_t cand_cap)
{
    for (int b = threadIdx.x; b < kRkBins2; b += kBlock) {
        reinterpret_cast<uint32_t*>(ws->hist1)[b] = 0u;  // kRkCopies * kRkBins1 == kRkBins2
        ws->hist2[b] = 0u;
    }
    if (threadIdx.x < sizeof(RandkControl) / 4) {
        uint32_t v = 0u;
        if (threadIdx.x == offsetof(RandkControl, x_lo) / 4)
            v = x_lo;
        if (threadIdx.x == offsetof(RandkControl, x_hi) / 4)
            v = x_hi;
        if (threadIdx.x == offsetof(RandkControl, cand_cap) / 4)
            v = cand_cap;
        reinterpret_cast<uint32_t*>(&ws->ctl)[threadIdx.x] = v;
    }
    if (threadIdx.x < kRkShards) {
        ws->n_stage[threadIdx.x][0] = 0u;
        ws->n_bcand[threadIdx.x][0] = 0u;
    }
}

// The kRkUnroll key groups q0 + u * kBlock (u < kRkUnroll) of one thread and
// iteration; groups at or past nq get an all-zero block and must be skipped.
__device__ __forceinline__ void key_blocks(int64_t q0, int64_t nq, uint32_t purpose, uint32_t key0, uint32_t key1,
                                           uint4 w[kRkUnroll])
{
#pragma unroll
    for (int u = 0; u < kRkUnroll; ++u) {
        const int64_t q = q0 + static_cast<int64_t>(u) * kBlock;
        w[u] = q < nq ? selection_block(static_cast<uint32_t>(q), purpose, key0, key1) : make_uint4(0u, 0u, 0u, 0u);
    }
}

// Pass 1: histogram of the top 8 bits of hi.
static_assert(kRkBins1 == kBlock, "one level-1 bin per thread");
__global__ __launch_bounds__(kBlock) void k_rk_hist1(int64_t d, uint32_t key0, uint32_t key1,
                                                     RandkWorkspace* __restrict__ ws)
{
    __shared__ uint32_t h[kRkBins1];
    h[threadIdx.x] = 0u;
    __syncthreads();
    const int64_t nq = (d + 3) >> 2;
    const int64_t step = static_cast<int64_t>(gridDim.x) * kBlock * kRkUnroll;
    for (int64_t q0 = static_cast<int64_t>(blockIdx.x) * kBlock * kRkUnroll + threadIdx.x; q0 < nq; q0 += step) {
        uint4 w[kRkUnroll];
        key_blocks(q0, nq, 2u, key0, key1, w);
#pragma unroll
        for (int u = 0; u < kRkUnroll; ++u) {
            const int64_t q = q0 + static_cast<int64_t>(u) * kBlock;
#pragma unroll
            for (int j = 0; j < 4; ++j)
                if ((q << 2) + j < d)
                    atomicAdd(&h[word_of(w[u], j) >> 24], 1u);
        }
    }
    __syncthreads();
    if (h[threadIdx.x] != 0u)
        atomicAdd(&ws->hist1[blockIdx.x % kRkCopies][threadIdx.x], h[threadIdx.x]);
}

// Pass 2: every block finds (b1, need1); keys in bin b1 histogram bits
// 23..12 of hi.
__global__ __launch_bounds__(kBlock) void k_rk_hist2(int64_t d, uint32_t K, uint32_t key0, uint32_t key1,
                                                     RandkWorkspace* __restrict__ ws)
{
    __shared__ uint32_t scratch[kBlock / 64];
    __shared__ uint32_t found[2];
    __shared__ uint32_t hist1[kRkBins1];
    uint32_t c[kRkCopies];
#pragma unroll
    for (int k = 0; k < kRkCopies; ++k)
        c[k] = ws->hist1[k][threadIdx.x];
    uint32_t total = 0u;
#pragma unroll
    for (int k = 0; k < kRkCopies; ++k)
        total += c[k];
    hist1[threadIdx.x] = total;
    __syncthreads();
    find_bin<1>(hist1, K, scratch, &found[0], &found[1]);
    __syncthreads();
    const uint32_t b1 = found[0];
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        ws->ctl.b1 = b1;
        ws->ctl.need1 = found[1];
    }
    const int64_t nq = (d + 3) >> 2;
    const int64_t step = static_cast<int64_t>(gridDim.x) * kBlock * kRkUnroll;
    for (int64_t q0 = static_cast<int64_t>(blockIdx.x) * kBlock * kRkUnroll + threadIdx.x; q0 < nq; q0 += step) {
        uint4 w[kRkUnroll];
        key_blocks(q0, nq, 2u, key0, key1, w);
#pragma unroll
        for (int u = 0; u < kRkUnroll; ++u) {
            const int64_t q = q0 + static_cast<int64_t>(u) * kBlock;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const uint32_t hi = word_of(w[u], j);
                if ((q << 2) + j < d && (hi >> 24) == b1)
                    atomicAdd(&ws->hist2[(hi >> 12) & 0xFFFu], 1u);
            }
        }
    }
}

// One block: the level-2 sub-bin b2 holding the need1-th key of bin b1; the
// collection interval is the keys with that 20-bit prefix.
__global__ __launch_bounds__(kBlock) void k_rk_scan2(RandkWorkspace* __restrict__ ws)
{
    __shared__ uint32_t scratch[kBlock / 64];
    __shared__ uint32_t found[2];
    find_bin<kRkBins2 / kBlock>(ws->hist2, ws->ctl.need1, scratch, &found[0], &found[1]);
    __syncthreads();
    if (threadIdx.x == 0) {
        ws->ctl.b2 = found[0];
        ws->ctl.need2 = found[1];
        ws->ctl.x_lo = (ws->ctl.b1 << 24) | (found[0] << 12);
        ws->ctl.x_hi = (ws->ctl.b1 << 24) | (found[0] << 12) | 0xFFFu;
    }
}

// Pass 3: collect the keys whose hi lies in [x_lo, x_hi], with low words.
// With PICK (K <= kRkSortMax) the keys below x_lo are appended to the staging
// lists in the same pass (all selected when the interval holds the K-th
// key): each wave adds its selections of a key group to list (wave id mod
// kRkShards) with one atomic.  SHARDED (the bracket, about 20 sqrt(K)
// candidates) puts the candidates in per-list arrays, so that their append
// counters are spread too; otherwise (d / 2^20 expected) they go to one list.
template <bool PICK, bool SHARDED>
__global__ __launch_bounds__(kBlock) void k_rk_collect(int64_t d, uint32_t key0, uint32_t key1,
                                                       RandkWorkspace* __restrict__ ws, uint32_t K)
{
    const uint32_t x_lo = ws->ctl.x_lo, x_hi = ws->ctl.x_hi;
    const int lane = threadIdx.x & 63;
    const uint64_t below_lanes = (uint64_t(1) << lane) - 1u;
    const uint32_t shard = (blockIdx.x * (kBlock / 64) + (threadIdx.x >> 6)) % kRkShards;
    uint32_t* list = ws->stage[shard];
    const int64_t nq = (d + 3) >> 2;
    const int64_t step = static_cast<int64_t>(gridDim.x) * kBlock * kRkUnroll;
    for (int64_t q0 = static_cast<int64_t>(blockIdx.x) * kBlock * kRkUnroll + threadIdx.x; q0 < nq; q0 += step) {
      uint4 wu[kRkUnroll];
      key_blocks(q0, nq, 2u, key0, key1, wu);
#pragma unroll
      for (int u = 0; u < kRkUnroll; ++u) {
        const int64_t q = q0 + static_cast<int64_t>(u) * kBlock;
        const uint4 w = wu[u];
        bool any = false;
        uint32_t take = 0u;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const bool in = (q << 2) + j < d;
            const uint32_t hi = word_of(w, j);
            any = any || (in && hi >= x_lo && hi <= x_hi);
            take |= (PICK && in && hi < x_lo) ? (1u << j) : 0u;
        }
        if (any) {
            const uint4 l = selection_block(static_cast<uint32_t>(q), 3u, key0, key1);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int64_t i = (q << 2) + j;
                if (i < d && word_of(w, j) >= x_lo && word_of(w, j) <= x_hi) {
                    if (SHARDED) {
                        const uint32_t slot = atomicAdd(&ws->n_bcand[shard][0], 1u);
                        if (slot < static_cast<uint32_t>(kRkShardCand)) {
                            ws->bcand[shard][slot][0] = word_of(w, j);
                            ws->bcand[shard][slot][1] = word_of(l, j);
                            ws->bcand[shard][slot][2] = static_cast<uint32_t>(i);
                        }
                    } else {
                        const uint32_t slot = atomicAdd(&ws->ctl.n_cand, 1u);
                        if (slot < ws->ctl.cand_cap) {
                            ws->cand[slot][0] = word_of(w, j);
                            ws->cand[slot][1] = word_of(l, j);
                            ws->cand[slot][2] = static_cast<uint32_t>(i);
                        }
                    }
                }
            }
        }
        if (PICK) {
            uint32_t before = 0u, total = 0u;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const uint64_t bal = __ballot((take >> j) & 1u);
                before += __popcll(bal & below_lanes);
                total += __popcll(bal);
            }
            if (total != 0u) {  // wave-uniform
                uint32_t base = 0u;
                if (lane == 0)
                    base = atomicAdd(&ws->n_stage[shard][0], total);
                base = __shfl(base, 0, 64);
                uint32_t pos = base + before;
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    if ((take >> j) & 1u) {
                        if (pos < K)  // at most K in all lists together; the guard keeps writes in bounds
                            list[pos] = static_cast<uint32_t>((q << 2) + j);
                        ++pos;
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

// One block, when the keys that share the K-th key's 20-bit prefix P did
// not all fit the candidate list: the need-th smallest (hi, lo, index) among
// them, exactly.  A histogram (in LDS, over every key) of the low 12 bits of
// hi among the keys with prefix P gives the K-th key's whole hi h* and how
// many keys with hi == h* are still needed; those keys (expected at most one
// or two for d < 2^32) are collected in LDS and ranked.  False (nothing
// written) only if more than `cap` keys share that 32-bit hi, which
// pseudo-random keys do not produce.
constexpr uint32_t kRkRefineCap = 1024;

template <int T>
__device__ bool refine_threshold(int64_t d, uint32_t key0, uint32_t key1, uint32_t P, uint32_t need, uint32_t* h,
                                 uint32_t (*cand)[3], uint32_t cap, uint32_t* scratch, uint32_t* found,
                                 uint32_t* th, uint32_t* tl, uint32_t* ti)
{
    const int64_t nq = (d + 3) >> 2;
    const uint32_t t = threadIdx.x;
    for (int b = t; b < kRkBins2; b += T)
        h[b] = 0u;
    __syncthreads();
    for (int64_t q = t; q < nq; q += T) {
        const uint4 w = selection_block(static_cast<uint32_t>(q), 2u, key0, key1);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const uint32_t hi = word_of(w, j);
            if ((q << 2) + j < d && (hi >> 12) == P)
                atomicAdd(&h[hi & 0xFFFu], 1u);
        }
    }
    __syncthreads();
    find_bin<kRkBins2 / T, T>(h, need, scratch, &found[0], &found[1]);
    __syncthreads();
    const uint32_t hstar = (P << 12) | found[0], need3 = found[1];
    __syncthreads();
    if (t == 0)
        found[0] = 0u;
    __syncthreads();
    for (int64_t q = t; q < nq; q += T) {
        const uint4 w = selection_block(static_cast<uint32_t>(q), 2u, key0, key1);
        bool any = false;
#pragma unroll
        for (int j = 0; j < 4; ++j)
            any = any || (((q << 2) + j < d) && word_of(w, j) == hstar);
        if (any) {
            const uint4 l = selection_block(static_cast<uint32_t>(q), 3u, key0, key1);
#pragma unroll
            for (int j = 0; j < 4; ++j)
                if (((q << 2) + j < d) && word_of(w, j) == hstar) {
                    const uint32_t slot = atomicAdd(&found[0], 1u);
                    if (slot < cap) {
                        cand[slot][0] = hstar;
                        cand[slot][1] = word_of(l, j);
                        cand[slot][2] = static_cast<uint32_t>((q << 2) + j);
                    }
                }
        }
    }
    __syncthreads();
    const uint32_t n = found[0];
    const bool ok = n <= cap;  // block-uniform
    if (ok) {
        for (uint32_t c = t; c < n; c += T) {
            uint32_t rank = 0u;
            for (uint32_t u = 0; u < n; ++u)
                rank += key_less(cand[u][0], cand[u][1], cand[u][2], cand[c][0], cand[c][1], cand[c][2]) ? 1u : 0u;
            if (rank == need3 - 1u) {
                *th = cand[c][0];
                *tl = cand[c][1];
                *ti = cand[c][2];
            }
        }
    }
    __syncthreads();
    return ok;
}

// One block: the candidate whose rank among the candidates (by hi, lo,
// index; all distinct) is need2 - 1 is the threshold.  About d / 2^20
// candidates are expected, so a direct count of smaller keys is cheapest.
// With PICK the candidates of rank below need2 (the selected ones) are
// appended to staging list 0.  If more candidates arrived than the list
// keeps, the threshold comes from refine_threshold instead and (with PICK)
// ctl.exact sends the sort to the exact path; should that fail too, every
// output entry is 0xFFFFFFFF and the later passes select nothing.
template <bool PICK>
__global__ __launch_bounds__(kRkSortThreads) void k_rk_threshold(RandkWorkspace* __restrict__ ws, uint32_t K,
                                                                 int64_t d, uint32_t key0, uint32_t key1,
                                                                 uint32_t* __restrict__ sel)
{
    __shared__ uint32_t h[kRkBins2];
    __shared__ uint32_t cand[kRkRefineCap][3];
    __shared__ uint32_t scratch[kRkSortThreads / 64];
    __shared__ uint32_t found[2];
    __shared__ uint32_t thr[3];
    const uint32_t n_all = ws->ctl.n_cand;
    const uint32_t want = ws->ctl.need2 - 1u;
    if (n_all > ws->ctl.cand_cap) {  // block-uniform
        const uint32_t P = (ws->ctl.b1 << 12) | ws->ctl.b2;
        const bool ok = refine_threshold<kRkSortThreads>(d, key0, key1, P, want + 1u, h, cand, kRkRefineCap,
                                                         scratch, found, &thr[0], &thr[1], &thr[2]);
        if (threadIdx.x == 0) {
            ws->ctl.exact = 1u;
            ws->ctl.thr_hi = ok ? thr[0] : 0u;
            ws->ctl.thr_lo = ok ? thr[1] : 0u;
            ws->ctl.thr_idx = ok ? thr[2] : 0u;
            if (!ok)
                ws->ctl.exact = 2u;
        }
        if (!ok)
            for (uint32_t j = threadIdx.x; j < K; j += kRkSortThreads)
                sel[j] = 0xFFFFFFFFu;
        return;
    }
    const uint32_t n = n_all;
    for (uint32_t t = threadIdx.x; t < n; t += kRkSortThreads) {
        const uint32_t h0 = ws->cand[t][0], l = ws->cand[t][1], i = ws->cand[t][2];
        uint32_t rank = 0u;
        for (uint32_t u = 0; u < n; ++u)
            rank += key_less(ws->cand[u][0], ws->cand[u][1], ws->cand[u][2], h0, l, i) ? 1u : 0u;
        if (rank == want) {
            ws->ctl.thr_hi = h0;
            ws->ctl.thr_lo = l;
            ws->ctl.thr_idx = i;
        }
        if (PICK && rank <= want) {
            const uint32_t pos = atomicAdd(&ws->n_stage[0][0], 1u);
            if (pos < K)
                ws->stage[0][pos] = i;
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

// ---------------------------------------------------------------------------
// Selection by a bracket.  The number of keys with hi < x is binomial,
// Binomial(d, x / 2^32), so the host can name an interval [x_lo, x_hi] of hi
// that holds the K-th key except with probability below 1e-20 (ten standard
// deviations either side); one collection pass then appends every key below
// x_lo to the staging lists and gathers the roughly 20 sqrt(K) keys inside
// the interval as candidates, and every block of the sort completes the
// selection for itself: it checks that the interval did hold the K-th key
// (fewer than K keys below it, at least K at or below its top, every
// candidate kept), cuts the interval into kRkPickBuckets equal parts counted
// in LDS, ranks the part where the count reaches K exactly and takes the parts
// before it whole.  If the check fails, the block computes the exact
// selection on its own, slowly (the histogram steps of the multi-pass path,
// then one pass that writes its slice of the output in order), so the result
// never depends on the bracket.
// ---------------------------------------------------------------------------
constexpr int kRkPickBuckets = 2048;  // the interval cut into equal parts
constexpr int kRkCross = 512;         // candidates of the crossing part kept in LDS
constexpr int kRkPickMax = 4096;      // bracket candidates a sort block holds in LDS

__device__ __forceinline__ uint32_t pick_bucket(uint32_t hi, uint32_t x_lo, uint64_t width)
{
    return static_cast<uint32_t>((static_cast<uint64_t>(hi - x_lo) * kRkPickBuckets) / width);
}

constexpr int kRkBuckets = 4 * kRkSortThreads;  // buckets of the index range in the sort

// Bucket of index i < d among kRkBuckets equal parts of [0, d): a monotone
// map, clamped so that no index can address outside the counters.
__device__ __forceinline__ uint32_t bucket_of(uint32_t i, double scale)
{
    const uint32_t b = static_cast<uint32_t>(static_cast<double>(i) * scale);
    return b < kRkBuckets ? b : kRkBuckets - 1u;
}

// The K staged indices in increasing order, by kRkSlices blocks.  The index
// range is cut into kRkBuckets buckets (a monotone map) and block j owns the
// contiguous run of buckets j * kRkSliceBuckets .. + kRkSliceBuckets - 1.
// Every block reads all staged indices (16 threads per staging list), counts
// those in earlier slices (its output offset) and bins its own through LDS
// counters (about K / kRkBuckets per bucket); a second read places them by
// bucket, and each is written at the offset plus its bucket's start plus its
// rank inside the bucket (the indices are distinct).
constexpr int kRkSlices = 64;
constexpr int kRkSliceBuckets = kRkBuckets / kRkSlices;
static_assert(kRkSliceBuckets == 64, "one wave scans a slice's buckets");
static_assert(kRkShards * 16 == kRkSortThreads, "16 threads per staging list");

// The selections of one block's slice of the output, in index order, given
// the threshold (th, tl, ti): one pass in index order that counts the
// selections of earlier slices (the slice's offset) and writes the slice's
// own at their places.
__device__ void write_slice_in_order(int64_t d, uint32_t K, uint32_t key0, uint32_t key1, uint32_t* __restrict__ sel,
                                     uint32_t th, uint32_t tl, uint32_t ti, uint32_t* scratch)
{
    constexpr int T = kRkSortThreads;
    const int64_t nq = (d + 3) >> 2;
    const uint32_t t = threadIdx.x;
    const uint32_t slice = blockIdx.x;
    const double scale = static_cast<double>(kRkBuckets) / static_cast<double>(d);
    uint32_t below = 0u, mine = 0u;
    for (int64_t qb = 0; qb < nq; qb += T) {
        // past the slice: nothing more to write (the bucket map is monotone)
        if (bucket_of(static_cast<uint32_t>(qb << 2), scale) / kRkSliceBuckets > slice)
            break;
        const int64_t q = qb + t;
        const uint32_t mask = q < nq ? selected_mask(q, d, key0, key1, th, tl, ti) : 0u;
        uint32_t mb = 0u, mm = 0u;
#pragma unroll
        for (int j = 0; j < 4; ++j)
            if ((mask >> j) & 1u) {
                const uint32_t sl = bucket_of(static_cast<uint32_t>((q << 2) + j), scale) / kRkSliceBuckets;
                mb |= sl < slice ? (1u << j) : 0u;
                mm |= sl == slice ? (1u << j) : 0u;
            }
        const uint32_t nb = __builtin_popcount(mb), nm = __builtin_popcount(mm);
        const uint32_t ib = block_inclusive_scan<T>(nb, scratch);
        if (t == T - 1)
            scratch[T / 64] = ib;
        __syncthreads();
        below += scratch[T / 64];  // earlier slices' selections have smaller indices
        __syncthreads();
        const uint32_t im = block_inclusive_scan<T>(nm, scratch);
        uint32_t pos = below + mine + im - nm;
#pragma unroll
        for (int j = 0; j < 4; ++j)
            if ((mm >> j) & 1u) {
                if (pos < K)
                    sel[pos] = static_cast<uint32_t>((q << 2) + j);
                ++pos;
            }
        if (t == T - 1)
            scratch[T / 64] = im;
        __syncthreads();
        mine += scratch[T / 64];
        __syncthreads();
    }
}

// The exact selection, for one block's slice of the output (the bracket
// missed): level-1 and level-2 histograms of hi in LDS, the candidates that
// share the K-th key's 20-bit prefix ranked for the threshold (key, index)
// (if more than `cap` of them arrive, refine_threshold finds it instead),
// then the slice written in order.  cand: LDS room for kRkSortMax / 3
// candidates (about d / 2^20 are expected, at most 4096 on average for
// d < 2^32).  Should refine_threshold fail, every output entry is 0xFFFFFFFF.
__device__ void sort_exact_slice(int64_t d, uint32_t K, uint32_t key0, uint32_t key1, uint32_t* __restrict__ sel,
                                 uint32_t* h, uint32_t (*cand)[3], uint32_t* scratch, uint32_t* found, uint32_t cap)
{
    constexpr int T = kRkSortThreads;
    constexpr uint32_t kCap = kRkSortMax / 3;
    cap = cap < kCap ? cap : kCap;
    const int64_t nq = (d + 3) >> 2;
    const uint32_t t = threadIdx.x;
    // level 1: hi >> 24
    for (int b = t; b < kRkBins2; b += T)
        h[b] = 0u;
    __syncthreads();
    for (int64_t q = t; q < nq; q += T) {
        const uint4 w = selection_block(static_cast<uint32_t>(q), 2u, key0, key1);
#pragma unroll
        for (int j = 0; j < 4; ++j)
            if ((q << 2) + j < d)
                atomicAdd(&h[word_of(w, j) >> 24], 1u);
    }
    __syncthreads();
    find_bin<kRkBins2 / T, T>(h, K, scratch, &found[0], &found[1]);  // bins past 255 are empty
    __syncthreads();
    const uint32_t b1 = found[0], need1 = found[1];
    __syncthreads();
    // level 2: (hi >> 12) & 0xFFF in bin b1
    for (int b = t; b < kRkBins2; b += T)
        h[b] = 0u;
    __syncthreads();
    for (int64_t q = t; q < nq; q += T) {
        const uint4 w = selection_block(static_cast<uint32_t>(q), 2u, key0, key1);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const uint32_t hi = word_of(w, j);
            if ((q << 2) + j < d && (hi >> 24) == b1)
                atomicAdd(&h[(hi >> 12) & 0xFFFu], 1u);
        }
    }
    __syncthreads();
    find_bin<kRkBins2 / T, T>(h, need1, scratch, &found[0], &found[1]);
    __syncthreads();
    const uint32_t prefix = (b1 << 12) | found[0], need2 = found[1];
    __syncthreads();
    if (t == 0)
        found[0] = 0u;  // candidate count
    __syncthreads();
    for (int64_t q = t; q < nq; q += T) {
        const uint4 w = selection_block(static_cast<uint32_t>(q), 2u, key0, key1);
        bool any = false;
#pragma unroll
        for (int j = 0; j < 4; ++j)
            any = any || (((q << 2) + j < d) && (word_of(w, j) >> 12) == prefix);
        if (any) {
            const uint4 l = selection_block(static_cast<uint32_t>(q), 3u, key0, key1);
#pragma unroll
            for (int j = 0; j < 4; ++j)
                if (((q << 2) + j < d) && (word_of(w, j) >> 12) == prefix) {
                    const uint32_t slot = atomicAdd(&found[0], 1u);
                    if (slot < cap) {
                        cand[slot][0] = word_of(w, j);
                        cand[slot][1] = word_of(l, j);
                        cand[slot][2] = static_cast<uint32_t>((q << 2) + j);
                    }
                }
        }
    }
    __syncthreads();
    const uint32_t n = found[0];
    __syncthreads();
    __shared__ uint32_t thr[3];
    if (n <= cap) {  // block-uniform
        for (uint32_t c = t; c < n; c += T) {
            uint32_t rank = 0u;
            for (uint32_t u = 0; u < n; ++u)
                rank += key_less(cand[u][0], cand[u][1], cand[u][2], cand[c][0], cand[c][1], cand[c][2]) ? 1u : 0u;
            if (rank == need2 - 1u) {
                thr[0] = cand[c][0];
                thr[1] = cand[c][1];
                thr[2] = cand[c][2];
            }
        }
        __syncthreads();
    } else if (!refine_threshold<T>(d, key0, key1, prefix, need2, h, cand, kRkRefineCap, scratch, found, &thr[0],
                                    &thr[1], &thr[2])) {
        for (uint32_t j = t; j < K; j += T)
            sel[j] = 0xFFFFFFFFu;
        return;
    }
    const uint32_t th = thr[0], tl = thr[1], ti = thr[2];
    __syncthreads();
    write_slice_in_order(d, K, key0, key1, sel, th, tl, ti, scratch);
}

// The staged indices (and, with BRACKET, the picks this block makes among
// the bracket's candidates) in increasing order, by kRkSlices blocks.  The
// index range is cut into kRkBuckets buckets (a monotone map) and block j owns
// the contiguous run of buckets j * kRkSliceBuckets .. + kRkSliceBuckets - 1.
// Every block reads all staged indices (16 threads per staging list), counts
// those in earlier slices (its output offset) and bins its own through LDS
// counters (about K / kRkBuckets per bucket); a second read places them by
// bucket, and each is written at the offset plus its bucket's start plus its
// rank inside the bucket (the indices are distinct).
template <bool BRACKET>
__global__ __launch_bounds__(kRkSortThreads) void k_rk_sort(const RandkWorkspace* __restrict__ ws,
                                                            uint32_t* __restrict__ sel, uint32_t K, int64_t d,
                                                            uint32_t key0, uint32_t key1)
{
    __shared__ uint32_t buf[kRkSortMax];
    __shared__ uint32_t count[kRkSliceBuckets];
    __shared__ uint32_t start[kRkSliceBuckets];
    __shared__ uint32_t wave_below[kRkSortThreads / 64];
    __shared__ uint32_t n_mine;
    const uint32_t t = threadIdx.x;
    const uint32_t slice = blockIdx.x;
    const int lane = t & 63, wave = t >> 6;
    const uint32_t* list = ws->stage[t >> 4];
    const uint32_t len = min(ws->n_stage[t >> 4][0], static_cast<uint32_t>(kRkSortMax));
    const uint32_t sub = t & 15u;
    const double scale = static_cast<double>(kRkBuckets) / static_cast<double>(d);

    // BRACKET: this block's picks among the candidates, in h[0 .. n_pick)
    __shared__ uint32_t h[BRACKET ? kRkBins2 : 1];
    __shared__ uint32_t cl[BRACKET ? kRkPickMax : 1][3];
    __shared__ uint32_t cross[BRACKET ? kRkCross : 1][3];
    __shared__ uint32_t scratch[kRkSortThreads / 64 + 4];
    __shared__ uint32_t found[2];
    __shared__ uint32_t n_list[kRkShards], list_off[kRkShards];
    __shared__ uint32_t n_cross, n_pick, overflow;
    uint32_t npick = 0u;
    if (BRACKET) {
        static_assert(kRkPickBuckets == 2 * kRkSortThreads, "two parts per thread in the scan");
        const uint32_t x_lo = ws->ctl.x_lo, x_hi = ws->ctl.x_hi;
        const uint64_t width = static_cast<uint64_t>(x_hi - x_lo) + 1u;
        if (t == 0) {
            n_cross = 0u;
            n_pick = 0u;
            overflow = 0u;
        }
        for (int b = t; b < kRkPickBuckets; b += kRkSortThreads)
            h[b] = 0u;
        __syncthreads();
        uint32_t below = 0u, cands = 0u;
        if (t < kRkShards) {
            below = ws->n_stage[t][0];
            cands = ws->n_bcand[t][0];
            n_list[t] = cands;
            if (cands > static_cast<uint32_t>(kRkShardCand))
                atomicOr(&overflow, 1u);
        }
        const uint32_t ib = block_inclusive_scan<kRkSortThreads>(below, scratch);
        if (t == kRkSortThreads - 1)
            found[0] = ib;  // the last thread's inclusive sum is the total
        const uint32_t ic = block_inclusive_scan<kRkSortThreads>(cands, scratch);
        if (t == kRkSortThreads - 1)
            found[1] = ic;
        if (t < kRkShards)
            list_off[t] = ic - cands;
        __syncthreads();
        const uint32_t staged = found[0];
        const uint32_t n_c = found[1];
        bool valid = overflow == 0u && n_c <= static_cast<uint32_t>(kRkPickMax) && staged < K && staged + n_c >= K;
        uint32_t bstar = 0u, rest = 0u;
        if (valid) {
            {  // gather: 16 threads per list
                const uint32_t sh = t >> 4, n = n_list[sh], off = list_off[sh];
                for (uint32_t j = sub; j < n; j += 16u) {
                    cl[off + j][0] = ws->bcand[sh][j][0];
                    cl[off + j][1] = ws->bcand[sh][j][1];
                    cl[off + j][2] = ws->bcand[sh][j][2];
                }
            }
            __syncthreads();
            for (uint32_t c = t; c < n_c; c += kRkSortThreads)
                atomicAdd(&h[pick_bucket(cl[c][0], x_lo, width)], 1u);
            __syncthreads();
            find_bin<kRkPickBuckets / kRkSortThreads, kRkSortThreads>(h, K - staged, scratch, &found[0], &found[1]);
            __syncthreads();
            bstar = found[0];
            rest = found[1];
            for (uint32_t c = t; c < n_c; c += kRkSortThreads)
                if (pick_bucket(cl[c][0], x_lo, width) == bstar) {
                    const uint32_t slot = atomicAdd(&n_cross, 1u);
                    if (slot < static_cast<uint32_t>(kRkCross)) {
                        cross[slot][0] = cl[c][0];
                        cross[slot][1] = cl[c][1];
                        cross[slot][2] = cl[c][2];
                    }
                }
            __syncthreads();
            valid = n_cross <= static_cast<uint32_t>(kRkCross);  // block-uniform
        }
        if (!valid) {
            sort_exact_slice(d, K, key0, key1, sel, h, reinterpret_cast<uint32_t(*)[3]>(buf), scratch, found,
                             ws->ctl.cand_cap);
            return;
        }
        // the picks, into h (the parts' counts are no longer needed)
        for (uint32_t c = t; c < n_c; c += kRkSortThreads) {
            const uint32_t hh = cl[c][0], ll = cl[c][1], ii = cl[c][2];
            const uint32_t b = pick_bucket(hh, x_lo, width);
            bool take = b < bstar;
            if (b == bstar) {
                uint32_t rank = 0u;
                for (uint32_t u = 0; u < n_cross; ++u)
                    rank += key_less(cross[u][0], cross[u][1], cross[u][2], hh, ll, ii) ? 1u : 0u;
                take = rank < rest;
            }
            if (take) {
                const uint32_t pos = atomicAdd(&n_pick, 1u);
                if (pos < static_cast<uint32_t>(kRkBins2))
                    h[pos] = ii;
            }
        }
        __syncthreads();
        npick = min(n_pick, static_cast<uint32_t>(kRkBins2));
    }

    if (!BRACKET && ws->ctl.exact != 0u) {
        // the histogram route's candidates overflowed: its threshold block
        // found the threshold exactly (or, failing, wrote the sentinel), but
        // the selected candidates were not staged, so the slice is written
        // from the keys themselves
        if (ws->ctl.exact == 1u)
            write_slice_in_order(d, K, key0, key1, sel, ws->ctl.thr_hi, ws->ctl.thr_lo, ws->ctl.thr_idx, scratch);
        return;
    }
    if (t < kRkSliceBuckets)
        count[t] = 0u;
    __syncthreads();
    uint32_t below = 0u;
#pragma unroll 4
    for (uint32_t p = sub; p < len; p += 16u) {
        const uint32_t b = bucket_of(list[p], scale);
        const uint32_t sl = b / kRkSliceBuckets;
        if (sl < slice)
            ++below;
        else if (sl == slice)
            atomicAdd(&count[b % kRkSliceBuckets], 1u);
    }
    for (uint32_t p = t; p < npick; p += kRkSortThreads) {
        const uint32_t b = bucket_of(h[p], scale);
        const uint32_t sl = b / kRkSliceBuckets;
        if (sl < slice)
            ++below;
        else if (sl == slice)
            atomicAdd(&count[b % kRkSliceBuckets], 1u);
    }
    // indices in earlier slices: the block's output offset
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1)
        below += __shfl_xor(below, off, 64);
    if (lane == 0)
        wave_below[wave] = below;
    __syncthreads();
    uint32_t offset = 0u;
#pragma unroll
    for (int v = 0; v < kRkSortThreads / 64; ++v)
        offset += wave_below[v];
    // exclusive scan of the slice's bucket counts (one wave, a bucket per lane)
    if (wave == 0) {
        const uint32_t c = count[lane];
        uint32_t x = c;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const uint32_t y = __shfl_up(x, off, 64);
            if (lane >= off)
                x += y;
        }
        start[lane] = x - c;
        if (lane == 63)
            n_mine = x;
        count[lane] = 0u;  // reused as the bucket's fill cursor
    }
    __syncthreads();
#pragma unroll 4
    for (uint32_t p = sub; p < len; p += 16u) {
        const uint32_t v = list[p];
        const uint32_t b = bucket_of(v, scale);
        if (b / kRkSliceBuckets == slice) {
            const uint32_t lb = b % kRkSliceBuckets;
            const uint32_t pos = start[lb] + atomicAdd(&count[lb], 1u);
            if (pos < static_cast<uint32_t>(kRkSortMax))
                buf[pos] = v;
        }
    }
    for (uint32_t p = t; p < npick; p += kRkSortThreads) {
        const uint32_t v = h[p];
        const uint32_t b = bucket_of(v, scale);
        if (b / kRkSliceBuckets == slice) {
            const uint32_t lb = b % kRkSliceBuckets;
            const uint32_t pos = start[lb] + atomicAdd(&count[lb], 1u);
            if (pos < static_cast<uint32_t>(kRkSortMax))
                buf[pos] = v;
        }
    }
    __syncthreads();
    // each of the slice's indices goes to the offset plus its bucket's start
    // plus the number of smaller indices in its bucket
    const uint32_t n = min(n_mine, static_cast<uint32_t>(kRkSortMax));
    for (uint32_t e = t; e < n; e += kRkSortThreads) {
        const uint32_t v = buf[e];
        const uint32_t lb = bucket_of(v, scale) % kRkSliceBuckets;
        const uint32_t s0 = start[lb];
        const uint32_t m = min(count[lb], static_cast<uint32_t>(kRkSortMax) - min(s0, static_cast<uint32_t>(kRkSortMax)));
        uint32_t rank = 0u;
        for (uint32_t a = 0; a < m; ++a)
            rank += buf[s0 + a] < v ? 1u : 0u;
        const uint32_t pos = offset + s0 + rank;
        if (pos < K)
            sel[pos] = v;
    }
}


// K > kRkSortMax: block b owns coordinates [b * chunk, (b + 1) * chunk); one
// pass counts its selections, the next writes them in order at the scanned
// offset.
__global__ __launch_bounds__(kBlock) void k_rk_count(int64_t d, int64_t chunk, uint32_t key0, uint32_t key1,
                                                     RandkWorkspace* __restrict__ ws)
{
    __shared__ uint32_t wave_count[kBlock / 64];
    const uint32_t th = ws->ctl.thr_hi, tl = ws->ctl.thr_lo, ti = ws->ctl.thr_idx;
    // the threshold could not be found (the output holds the sentinel): select nothing
    const int64_t q0 = ws->ctl.exact == 2u ? 0 : (static_cast<int64_t>(blockIdx.x) * chunk) >> 2;
    const int64_t q1 = ws->ctl.exact == 2u ? 0 : min((static_cast<int64_t>(blockIdx.x) + 1) * chunk, d + 3) >> 2;
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

// One block: exclusive scan of the per-block counts (thread t owns blocks
// [t * PER, (t + 1) * PER)).
__global__ __launch_bounds__(kBlock) void k_rk_offsets(RandkWorkspace* __restrict__ ws, int32_t nblocks)
{
    constexpr int PER = kRkMaxBlocks / kBlock;
    __shared__ uint32_t scratch[kBlock / 64];
    uint32_t v[PER];
    uint32_t s = 0u;
#pragma unroll
    for (int j = 0; j < PER; ++j) {
        const int b = threadIdx.x * PER + j;
        v[j] = b < nblocks ? ws->block_count[b] : 0u;
        s += v[j];
    }
    uint32_t run = block_inclusive_scan(s, scratch) - s;
#pragma unroll
    for (int j = 0; j < PER; ++j) {
        const int b = threadIdx.x * PER + j;
        if (b < nblocks)
            ws->block_offset[b] = run;
        run += v[j];
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
    const int64_t q0 = ws->ctl.exact == 2u ? 0 : (static_cast<int64_t>(blockIdx.x) * chunk) >> 2;
    const int64_t q1 = ws->ctl.exact == 2u ? 0 : min((static_cast<int64_t>(blockIdx.x) + 1) * chunk, d + 3) >> 2;
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

// Persistent grid for the key passes: kBlock * kRkUnroll key groups per block
// and iteration, at most eight blocks per compute unit.
static unsigned key_grid(int64_t d)
{
    const int64_t groups = (d + 3) >> 2;
    int64_t blocks = (groups + kBlock * kRkUnroll - 1) / (kBlock * kRkUnroll);
    const int64_t cap = grid_cap() / 8;
    blocks = blocks < 1 ? 1 : (blocks > cap ? cap : blocks);
    return static_cast<unsigned>(blocks);
}

static std::atomic<int32_t> g_randk_mode{kRandkBracket};

bool set_randk_mode(int32_t mode)
{
    if (mode < kRandkHistogram || mode > kRandkBracketMissNoCandidates)
        return false;
    g_randk_mode.store(mode, std::memory_order_relaxed);
    return true;
}

// The bracket [x_lo, x_hi] of hi for the K-th key (see k_rk_sort): the count
// of keys with hi < x has mean d x / 2^32 and standard deviation at most
// sqrt(K (1 - K / d)) near the K-th key; ten of those (plus one) either side
// of K.  False when the expected candidates would not fit.
static bool randk_bracket(int64_t d, int64_t K, uint32_t* x_lo, uint32_t* x_hi)
{
    const double dd = static_cast<double>(d), kk = static_cast<double>(K);
    const double sd = std::sqrt(kk * (1.0 - kk / dd)) + 1.0;
    const double span = 4294967296.0;
    double a = std::floor((kk - 10.0 * sd - 1.0) / dd * span);
    double b = std::ceil((kk + 10.0 * sd + 1.0) / dd * span);
    a = a < 0.0 ? 0.0 : a;
    b = b > span - 1.0 ? span - 1.0 : b;
    if (a > b)
        return false;
    const double expected = dd * (b - a + 1.0) / span;
    if (expected + 10.0 * std::sqrt(expected) + 16.0 > static_cast<double>(kRkPickMax))
        return false;
    *x_lo = static_cast<uint32_t>(a);
    *x_hi = static_cast<uint32_t>(b);
    return true;
}

hipError_t launch_randk_select(int64_t d, int64_t K, uint64_t seed, uint32_t* sel, void* ws_raw, hipStream_t stream)
{
    RandkWorkspace* ws = static_cast<RandkWorkspace*>(ws_raw);
    const uint32_t key0 = static_cast<uint32_t>(seed);
    const uint32_t key1 = static_cast<uint32_t>(seed >> 32);
    const unsigned gx = key_grid(d);  // persistent grid for the key passes
    const int32_t mode = g_randk_mode.load(std::memory_order_relaxed);
    // the test modes keep no candidates, so that the exact refinement runs
    const uint32_t cand_cap = (mode == kRandkHistogramNoCandidates || mode == kRandkBracketMissNoCandidates)
                                  ? 0u
                                  : static_cast<uint32_t>(kRandkCandidates);
    const bool histogram = mode == kRandkHistogram || mode == kRandkHistogramNoCandidates;
    uint32_t x_lo = 0u, x_hi = 0u;
    if (K <= kRkSortMax && !histogram && randk_bracket(d, K, &x_lo, &x_hi)) {
        if (mode == kRandkBracketMiss || mode == kRandkBracketMissNoCandidates)
            x_lo = x_hi = 0u;  // an interval that cannot hold the K-th key: the exact fallback runs
        hipLaunchKernelGGL(k_rk_init, dim3(1), dim3(kBlock), 0, stream, ws, x_lo, x_hi, cand_cap);
        hipLaunchKernelGGL((k_rk_collect<true, true>), dim3(gx), dim3(kBlock), 0, stream, d, key0, key1, ws,
                           static_cast<uint32_t>(K));
        hipLaunchKernelGGL((k_rk_sort<true>), dim3(kRkSlices), dim3(kRkSortThreads), 0, stream, ws, sel,
                           static_cast<uint32_t>(K), d, key0, key1);
        return hipGetLastError();
    }
    hipLaunchKernelGGL(k_rk_init, dim3(1), dim3(kBlock), 0, stream, ws, 0u, 0u, cand_cap);
    // the first histogram merges its LDS bins into global memory: few,
    // long-lived blocks keep those atomics to a few per bin
    int64_t hist_blocks = grid_cap() / 32;  // two blocks per compute unit
    hist_blocks = hist_blocks > static_cast<int64_t>(gx) ? static_cast<int64_t>(gx) : hist_blocks;
    hipLaunchKernelGGL(k_rk_hist1, dim3(static_cast<unsigned>(hist_blocks)), dim3(kBlock), 0, stream, d, key0, key1,
                       ws);
    hipLaunchKernelGGL(k_rk_hist2, dim3(gx), dim3(kBlock), 0, stream, d, static_cast<uint32_t>(K), key0, key1, ws);
    hipLaunchKernelGGL(k_rk_scan2, dim3(1), dim3(kBlock), 0, stream, ws);
    if (K <= kRkSortMax) {
        // the collection pass also appends the keys below the boundary
        // prefix; the threshold block appends the selected candidates
        hipLaunchKernelGGL((k_rk_collect<true, false>), dim3(gx), dim3(kBlock), 0, stream, d, key0, key1, ws,
                           static_cast<uint32_t>(K));
        hipLaunchKernelGGL(k_rk_threshold<true>, dim3(1), dim3(kRkSortThreads), 0, stream, ws,
                           static_cast<uint32_t>(K), d, key0, key1, sel);
        hipLaunchKernelGGL((k_rk_sort<false>), dim3(kRkSlices), dim3(kRkSortThreads), 0, stream, ws, sel,
                           static_cast<uint32_t>(K), d, key0, key1);
        return hipGetLastError();
    }
    hipLaunchKernelGGL((k_rk_collect<false, false>), dim3(gx), dim3(kBlock), 0, stream, d, key0, key1, ws,
                       static_cast<uint32_t>(K));
    hipLaunchKernelGGL(k_rk_threshold<false>, dim3(1), dim3(kRkSortThreads), 0, stream, ws,
                       static_cast<uint32_t>(K), d, key0, key1, sel);
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
