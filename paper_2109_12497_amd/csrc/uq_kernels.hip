// HIP kernels of libuq for MI355X (gfx950).
//
// The aggregation step of Algorithm 1 / Algorithm 2 (Sec. 3.1-3.2) as
// streaming kernels, each bound by HBM bandwidth:
//   k_sumsq      per-row, per-chunk fp64 sums of squares        (norm, pass 1)
//   k_finish     fixed-order reduction of the chunk sums, max    (norm, pass 2)
//                over rows, sqrt -> W
//   k_index      shared scale index from the largest |g| over    (Eq. (11) +
//                the workers at each coordinate                    sharing)
//   k_norm_max   several scales, 2..16 rows: the norm's tile     (norm + the
//                sums and the largest |g| over the rows in one     index's input)
//                read of the gradients
//   k_rowsum     sums of those tile sums
//   k_index_prep the rows' sums, W and the index pass's thresholds
//                and exponent table, once per call
//   k_index_max  the shared index from the maxima's keys
//   k_quantise   Philox draws + stochastic rounding + int8 pack  (Eq. (8)/(12))
//   k_sum        int8 (or 4-/2-bit) code rows -> int32           (all-reduce)
//                sums, optionally with the reconstruction applied  (+ Eq. (9)/(13))
//   k_quant_sum  the quantiser's codes added straight into the   (Eq. (8)/(12) +
//                int32 sums, never stored (+ the reconstruction)   all-reduce)
//   k_index_quant_sum  all of up to 16 rows held at once: the     (Eq. (11) +
//                shared index from their exact maxima, then        sharing, (12),
//                k_quant_sum's codes, sums and reconstruction      sum, (13))
//   k_quant_sum_split  one scale, 5 to 16 rows: a tile's rows     (Eq. (8),
//                split over a block's waves, their sums meeting    sum, (9))
//                in LDS
//   k_dequant    int32 (+ index) -> fp32                          (Eq. (9)/(13))
//
// Every per-coordinate result is a pure function of its inputs and the
// coordinate index, so the output is independent of the launch geometry;
// the norm's reduction tree depends only on d (and on which norm pass runs).
#include <atomic>

#include "uq_device.hpp"
#include "uq_launch.hpp"

namespace uq {

// ---------------------------------------------------------------------------
// Norm, pass 1: block (c, m) sums g[m][c*chunk .. min(d, (c+1)*chunk)) squared
// in binary64 (each square exact) and stores the partial in part[m*nchunks+c].
// chunk is a multiple of 1024, so every chunk starts 16-byte aligned.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kBlock) void k_sumsq(const float* __restrict__ g, int64_t d, int32_t M,
                                                  int64_t ldg, int64_t chunk, int32_t nchunks,
                                                  double* __restrict__ part)
{
    __shared__ double wave_part[kBlock / 64];
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int32_t c = blockIdx.x;
    const int64_t begin = static_cast<int64_t>(c) * chunk;
    const int64_t end = begin + chunk < d ? begin + chunk : d;
    const int64_t nvec = (end - begin) >> 2;
    // grid.y covers the rows (more rows than grid.y: the blocks take them in turn)
    for (int32_t m = blockIdx.y; m < M; m += gridDim.y) {
        const float* row = g + static_cast<int64_t>(m) * ldg;
        const float* v4 = row + begin;
        double acc0 = 0.0, acc1 = 0.0, acc2 = 0.0, acc3 = 0.0;
        int64_t j = threadIdx.x;
        for (; j + 3 * kBlock < nvec; j += 4 * kBlock) {
            const f32x4 a = load_nt(v4 + 4 * j);
            const f32x4 b = load_nt(v4 + 4 * (j + kBlock));
            const f32x4 e = load_nt(v4 + 4 * (j + 2 * kBlock));
            const f32x4 f = load_nt(v4 + 4 * (j + 3 * kBlock));
            acc0 = fma((double)a.x, (double)a.x, acc0); acc1 = fma((double)a.y, (double)a.y, acc1);
            acc2 = fma((double)a.z, (double)a.z, acc2); acc3 = fma((double)a.w, (double)a.w, acc3);
            acc0 = fma((double)b.x, (double)b.x, acc0); acc1 = fma((double)b.y, (double)b.y, acc1);
            acc2 = fma((double)b.z, (double)b.z, acc2); acc3 = fma((double)b.w, (double)b.w, acc3);
            acc0 = fma((double)e.x, (double)e.x, acc0); acc1 = fma((double)e.y, (double)e.y, acc1);
            acc2 = fma((double)e.z, (double)e.z, acc2); acc3 = fma((double)e.w, (double)e.w, acc3);
            acc0 = fma((double)f.x, (double)f.x, acc0); acc1 = fma((double)f.y, (double)f.y, acc1);
            acc2 = fma((double)f.z, (double)f.z, acc2); acc3 = fma((double)f.w, (double)f.w, acc3);
        }
        for (; j < nvec; j += kBlock) {
            const f32x4 a = load_nt(v4 + 4 * j);
            acc0 = fma((double)a.x, (double)a.x, acc0); acc1 = fma((double)a.y, (double)a.y, acc1);
            acc2 = fma((double)a.z, (double)a.z, acc2); acc3 = fma((double)a.w, (double)a.w, acc3);
        }
        // at most three trailing coordinates (only in the last chunk when d % 4 != 0)
        const int64_t tail = begin + (nvec << 2) + threadIdx.x;
        if (tail < end) {
            const double x = row[tail];
            acc0 = fma(x, x, acc0);
        }
        const double s = wave_sum((acc0 + acc1) + (acc2 + acc3));
        if (lane == 0)
            wave_part[wave] = s;
        __syncthreads();
        if (threadIdx.x == 0)
            part[static_cast<int64_t>(m) * nchunks + c] = (wave_part[0] + wave_part[1]) + (wave_part[2] + wave_part[3]);
        __syncthreads();  // wave_part is reused for the next row
    }
}

// ---------------------------------------------------------------------------
// Norm, pass 2 (one block of kFinishThreads): S_m = fixed-order sum of row m's
// chunk partials (lane-strided sequential sums, then a fixed butterfly), one
// wave per row (16 rows at once); W = RN32(sqrt(max_m S_m)), NaN if any S_m
// is NaN.
// ---------------------------------------------------------------------------
constexpr int kFinishThreads = 1024;

__global__ __launch_bounds__(kFinishThreads) void k_finish(const double* __restrict__ part, int32_t nchunks,
                                                           int32_t M, float* __restrict__ w)
{
    __shared__ double wave_best[kFinishThreads / 64];
    __shared__ int wave_nan[kFinishThreads / 64];
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    double best = 0.0;
    bool any_nan = false;
    for (int32_t m = wave; m < M; m += kFinishThreads / 64) {
        // nchunks <= 1024: at most 16 partials per lane, all loads in flight at once
        const double* p = part + static_cast<int64_t>(m) * nchunks;
        double x[16];
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            const int32_t c = lane + 64 * j;
            x[j] = c < nchunks ? p[c] : 0.0;
        }
        double s = 0.0;
#pragma unroll
        for (int j = 0; j < 16; ++j)
            s += x[j];
        const double S = wave_sum(s);
        any_nan = any_nan || (S != S);
        best = S > best ? S : best;
    }
    if (lane == 0) {
        wave_best[wave] = best;
        wave_nan[wave] = any_nan ? 1 : 0;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        double b = 0.0;
        int nan = 0;
        for (int i = 0; i < kFinishThreads / 64; ++i) {
            b = wave_best[i] > b ? wave_best[i] : b;
            nan |= wave_nan[i];
        }
        *w = nan ? __builtin_nanf("") : static_cast<float>(sqrt(b));
    }
}

// ---------------------------------------------------------------------------
// Shared scale index.  The per-worker rule (largest k with
// RN32(|g| inv_k) <= s_0) is non-increasing in |g|, so the minimum over the
// workers is the rule applied to the largest usable |g| at the coordinate;
// a coordinate with no usable |g| (all zero / non-finite) takes K-1.
// Four coordinates per thread per step, float4 loads over the M rows.
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t index_of(float amax, const float* inv, int32_t K, float s0,
                                             bool zero)
{
    if (zero || !(amax > 0.0f))
        return static_cast<uint32_t>(K - 1);
    int32_t count = 0;
#pragma unroll
    for (int k = 0; k < kMaxScales; ++k)
        if (k < K)
            count += (amax * inv[k] <= s0) ? 1 : 0;
    return static_cast<uint32_t>(count > 0 ? count - 1 : 0);
}

__device__ __forceinline__ float usable_or_zero(float v)
{
    const float a = fabsf(v);
    return a <= kFloatMax ? a : 0.0f;  // NaN compares false -> 0
}

// Largest usable |g| over the M rows at quad q.
__device__ __forceinline__ f32x4 rows_amax(const float* __restrict__ g, int64_t q, int32_t M, int64_t ldg)
{
    f32x4 amax = {0.0f, 0.0f, 0.0f, 0.0f};
    const float* p = g + (q << 2);
    for (int32_t m = 0; m < M; ++m) {
        const f32x4 v = load_nt(p + static_cast<int64_t>(m) * ldg);
        amax.x = fmaxf(amax.x, usable_or_zero(v.x));
        amax.y = fmaxf(amax.y, usable_or_zero(v.y));
        amax.z = fmaxf(amax.z, usable_or_zero(v.z));
        amax.w = fmaxf(amax.w, usable_or_zero(v.w));
    }
    return amax;
}

// NIB: the index stored as 4-bit fields, two coordinates a byte (the low
// nibble first); a quad's four fields are one 16-bit store.
template <bool NIB>
__global__ __launch_bounds__(kBlock) void k_index(const float* __restrict__ g, int64_t d, int32_t M,
                                                  int64_t ldg, const float* __restrict__ wptr,
                                                  ScaleSet S, uint8_t* __restrict__ idx)
{
    __shared__ float inv_s[kMaxScales];
    const int64_t nquad = d >> 2;
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock;
    const int64_t first = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
    // the maxima do not need W: the first quad's loads go out before the
    // tables are formed
    f32x4 amax0 = {0.0f, 0.0f, 0.0f, 0.0f};
    if (first < nquad)
        amax0 = rows_amax(g, first, M, ldg);

    const float W = *wptr;
    if (threadIdx.x < S.K)
        inv_s[threadIdx.x] = div_rn32(S.s[threadIdx.x], W);
    __syncthreads();
    float inv[kMaxScales];
#pragma unroll
    for (int k = 0; k < kMaxScales; ++k)
        inv[k] = k < S.K ? __builtin_bit_cast(float, __builtin_amdgcn_readfirstlane(
                                 __builtin_bit_cast(int, inv_s[k])))
                         : 0.0f;
    const bool zero = zero_path(W, inv[0]);
    const float s0 = S.s[0];
    const int32_t K = S.K;

    for (int64_t q = first; q < nquad; q += stride) {
        const f32x4 amax = q == first ? amax0 : rows_amax(g, q, M, ldg);
        const int sh = NIB ? 4 : 8;
        const uint32_t packed = index_of(amax.x, inv, K, s0, zero) |
                                (index_of(amax.y, inv, K, s0, zero) << sh) |
                                (index_of(amax.z, inv, K, s0, zero) << (2 * sh)) |
                                (index_of(amax.w, inv, K, s0, zero) << (3 * sh));
        if (NIB)
            *reinterpret_cast<uint16_t*>(idx + (q << 1)) = static_cast<uint16_t>(packed);
        else
            *reinterpret_cast<uint32_t*>(idx + (q << 2)) = packed;
    }
    // trailing d % 4 coordinates (with 4-bit fields one thread forms their
    // bytes, which two coordinates share)
    const int64_t t = (nquad << 2) + static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
    if (blockIdx.x == 0 && t < d && (!NIB || threadIdx.x == 0)) {
        uint32_t nib = 0u;
        for (int64_t i = t; i < (NIB ? d : t + 1); ++i) {
            float amax = 0.0f;
            for (int32_t m = 0; m < M; ++m)
                amax = fmaxf(amax, usable_or_zero(g[static_cast<int64_t>(m) * ldg + i]));
            const uint32_t v = index_of(amax, inv, K, s0, zero);
            if (!NIB) {
                idx[i] = static_cast<uint8_t>(v);
            } else {
                nib |= v << (4 * ((i - t) & 1));
                if (((i - t) & 1) || i + 1 == d) {
                    idx[i >> 1] = static_cast<uint8_t>(nib);
                    nib = 0u;
                }
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Fused shared scale for several scales and at most kFuseRows rows: one pass
// over the gradients forms the rows' tile sums of squares and, at every
// coordinate, bits 30..15 of the largest usable |g| over the rows (a key,
// uint16 [d] in the workspace); the index pass then reads the keys
// instead of the M rows, and the rows of the rare coordinates whose key
// equals a threshold's.
//   k_norm_max   block t: tile t of every row (below)
//   k_rowsum     block (b, m) sums partials [b s, (b + 1) s) of row m in a
//                fixed order (s = kRowsumSpan)
//   k_index_prep one block: those sums into S_m (the same order), W (the
//                rule of k_finish), the thresholds, their keys and the
//                exponent table, into the workspace
//   k_index_max  the index of every coordinate from its key and that table
// ---------------------------------------------------------------------------
// Barrier for LDS traffic only: the block's LDS writes are complete and
// visible, while its global loads and stores stay in flight (__syncthreads
// would also wait for those).
__device__ __forceinline__ void sync_lds()
{
    __asm__ volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Tile t = the whole quads [256 t, 256 t + 256) (coordinates 1024 t ..) of
// every row; one block per tile, and one more block for the d % 4 trailing
// coordinates, which have a partial of their own (on a grid capped below
// that, blocks stride over the tiles, each tile still with its own partials,
// so the reduction tree does not depend on the grid).  Wave w owns rows
// w, w + 4, ... (ROWS / 4 of them; rows past M re-read row M - 1 and are not
// accumulated): lane l loads quads l, l + 64, l + 128, l + 192 of the tile from
// each of its rows (4 KiB per row per wave), all loads issued at once.  The
// waves' maxima meet in LDS and leave as one coalesced store of their 16-bit
// keys; each row's squares leave as one fp64 partial per tile.  Measured at
// 2^30 coordinates and 16 rows (MI355X), with fp32 maxima then: 12.3 ms
// (0.74 of 8 TB/s) in a probe of this form,
// against 13.8 ms for blocks that loop over 16 tiles with the next tile's
// loads issued before the current tile's store, and 12.8-13.8 ms for every
// looping form tried (double-buffered, no prefetch, 8 waves of 2 rows,
// straight-line runs of 2 to 16 tiles): in them the maxima stores cost about
// 3.7 ms over a pass without them, here 1.3 ms.  The trailing coordinates
// have their own block so that their code adds no registers to the tiles'
// (102 registers with it, four waves per SIMD instead of five).
// The d % 4 trailing coordinates of every row (partial t = ntiles): each
// wave adds its own rows' squares; wave 0 forms the maximum over all rows.
template <int ROWS>
__device__ __forceinline__ void norm_max_tail(const float* __restrict__ g, int64_t d, int32_t M, int64_t ldg,
                                              int64_t ntiles, double* __restrict__ part, uint16_t* __restrict__ keys)
{
    constexpr int RPW = ROWS / 4;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int64_t tail = ((d >> 2) << 2) + lane;
    const int64_t nparts = ntiles + 1;
#pragma unroll
    for (int r = 0; r < RPW; ++r) {
        const int m = wave + 4 * r;
        const double x = tail < d ? g[static_cast<int64_t>(m < M ? m : M - 1) * ldg + tail] : 0.0;
        const double sum = wave_sum(x * x);
        if (lane == 0 && m < M)
            part[static_cast<int64_t>(m) * nparts + ntiles] = sum;
    }
    if (wave == 0 && tail < d) {
        float mt = 0.0f;
        for (int32_t m = 0; m < M; ++m)
            mt = fmaxf(mt, usable_or_zero(g[static_cast<int64_t>(m) * ldg + tail]));
        keys[tail] = static_cast<uint16_t>(__builtin_bit_cast(uint32_t, mt) >> 15);
    }
}

// Tile t < ntiles: its maxima's keys and the rows' partials t.
template <int ROWS, bool NT>
__device__ __forceinline__ void norm_max_tile(const float* __restrict__ g, int64_t d, int32_t M, int64_t ldg,
                                              int64_t ntiles, int64_t t, double* __restrict__ part,
                                              uint16_t* __restrict__ keys, f32x4 (*wave_max)[kBlock])
{
    constexpr int RPW = ROWS / 4;  // rows per wave
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int64_t nquad = d >> 2;
    const int64_t q0 = t * kBlock;  // first quad of the tile
    const int64_t qe = q0 + kBlock < nquad ? q0 + kBlock : nquad;  // > q0
    // quads past qe re-read quad qe - 1 (the loads carry no branch) and are
    // zeroed below
    f32x4 v[RPW][4];
#pragma unroll
    for (int r = 0; r < RPW; ++r) {
        const int m = wave + 4 * r;
        const float* row = g + static_cast<int64_t>(m < M ? m : M - 1) * ldg;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int64_t q = q0 + lane + 64 * j;
            v[r][j] = load_nt(row + ((q < qe ? q : qe - 1) << 2));
        }
    }
    f32x4 mx[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        mx[j] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
        if (q0 + lane + 64 * j >= qe) {
#pragma unroll
            for (int r = 0; r < RPW; ++r)
                v[r][j] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
        }
    }
    double acc[RPW];
#pragma unroll
    for (int r = 0; r < RPW; ++r) {
        double a = 0.0;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            a = fma((double)v[r][j].x, (double)v[r][j].x, a);
            a = fma((double)v[r][j].y, (double)v[r][j].y, a);
            a = fma((double)v[r][j].z, (double)v[r][j].z, a);
            a = fma((double)v[r][j].w, (double)v[r][j].w, a);
            mx[j].x = fmaxf(mx[j].x, usable_or_zero(v[r][j].x));
            mx[j].y = fmaxf(mx[j].y, usable_or_zero(v[r][j].y));
            mx[j].z = fmaxf(mx[j].z, usable_or_zero(v[r][j].z));
            mx[j].w = fmaxf(mx[j].w, usable_or_zero(v[r][j].w));
        }
        acc[r] = a;
    }
#pragma unroll
    for (int j = 0; j < 4; ++j)
        wave_max[wave][lane + 64 * j] = mx[j];
    sync_lds();
    const f32x4 m0 = wave_max[0][threadIdx.x], m1 = wave_max[1][threadIdx.x];
    const f32x4 m2 = wave_max[2][threadIdx.x], m3 = wave_max[3][threadIdx.x];
    sync_lds();  // wave_max is reused by the block's next tile
    const int64_t q = q0 + threadIdx.x;
    if (q < qe) {
        f32x4 o;
        o.x = fmaxf(fmaxf(m0.x, m1.x), fmaxf(m2.x, m3.x));
        o.y = fmaxf(fmaxf(m0.y, m1.y), fmaxf(m2.y, m3.y));
        o.z = fmaxf(fmaxf(m0.z, m1.z), fmaxf(m2.z, m3.z));
        o.w = fmaxf(fmaxf(m0.w, m1.w), fmaxf(m2.w, m3.w));
        // the keys: bits 30..15 of the four maxima (exponent and 8 mantissa
        // bits; the sign bit of a maximum is 0), two to a word.
        // __float_as_uint takes the component's value; __builtin_bit_cast of
        // a vector component compiled to a read of component x here.
        u32x2 k;
        k.x = (__float_as_uint(o.x) >> 15) | ((__float_as_uint(o.y) << 1) & 0xFFFF0000u);
        k.y = (__float_as_uint(o.z) >> 15) | ((__float_as_uint(o.w) << 1) & 0xFFFF0000u);
        u32x2* dst = reinterpret_cast<u32x2*>(keys + (q << 2));
        if (NT)
            __builtin_nontemporal_store(k, dst);
        else
            *dst = k;
    }
#pragma unroll
    for (int r = 0; r < RPW; ++r) {
        const double sum = wave_sum(acc[r]);
        const int m = wave + 4 * r;
        if (lane == 0 && m < M)
            part[static_cast<int64_t>(m) * (ntiles + 1) + t] = sum;
    }
}

// ONE: one block per tile plus the trailing coordinates' block (no loop);
// otherwise blocks stride over them.
template <int ROWS, bool NT, bool ONE>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(5))) void k_norm_max(const float* __restrict__ g, int64_t d, int32_t M,
                                                     int64_t ldg, int64_t ntiles, double* __restrict__ part,
                                                     uint16_t* __restrict__ keys)
{
    __shared__ f32x4 wave_max[4][kBlock];
    if (ONE) {
        const int64_t t = blockIdx.x;
        if (t < ntiles)
            norm_max_tile<ROWS, NT>(g, d, M, ldg, ntiles, t, part, keys, wave_max);
        else if (t == ntiles)
            norm_max_tail<ROWS>(g, d, M, ldg, ntiles, part, keys);
        return;
    }
    for (int64_t t = blockIdx.x; t < ntiles; t += gridDim.x)
        norm_max_tile<ROWS, NT>(g, d, M, ldg, ntiles, t, part, keys, wave_max);
    if (blockIdx.x == gridDim.x - 1)
        norm_max_tail<ROWS>(g, d, M, ldg, ntiles, part, keys);
}

// The block's fixed-order sum of p[b0, b1): lane-strided sequential sums
// (16 loads in flight per thread), a fixed butterfly, then the four waves in
// order.  The total is valid in thread 0; wave_part must not be reused before
// the block's next barrier.
__device__ __forceinline__ double rowsum_span(const double* __restrict__ p, int64_t b0, int64_t b1,
                                              double* wave_part)
{
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    double s = 0.0;
    for (int64_t j0 = b0; j0 < b1; j0 += 16 * kBlock) {
        double x[16];
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            const int64_t c = j0 + static_cast<int64_t>(threadIdx.x) + kBlock * j;
            x[j] = c < b1 ? p[c] : 0.0;
        }
#pragma unroll
        for (int j = 0; j < 16; ++j)
            s += x[j];
    }
    s = wave_sum(s);
    if (lane == 0)
        wave_part[wave] = s;
    __syncthreads();
    return (wave_part[0] + wave_part[1]) + (wave_part[2] + wave_part[3]);
}

// Block (b, m) sums part[m][b * span .. min(n, (b + 1) * span)) in the fixed
// order of rowsum_span into out[m * gridDim.x + b].
__global__ __launch_bounds__(kBlock) void k_rowsum(const double* __restrict__ part, int64_t n, int64_t span,
                                                   double* __restrict__ out)
{
    __shared__ double wave_part[kBlock / 64];
    const int64_t b0 = static_cast<int64_t>(blockIdx.x) * span;
    const int64_t b1 = b0 + span < n ? b0 + span : n;
    const double s = rowsum_span(part + static_cast<int64_t>(blockIdx.y) * n, b0, b1, wave_part);
    if (threadIdx.x == 0)
        out[static_cast<int64_t>(blockIdx.y) * gridDim.x + blockIdx.x] = s;
}

// k_index_max: a block covers kIndexTile octets of coordinates (4 per
// thread: octets t, t + 256, ..., so each load and store of a wave is
// contiguous), all loaded before the call's constants are read.  The norm
// pass keeps, for each
// coordinate, bits 30..15 of its largest usable |g| over the rows (a key:
// the exponent field and the top 8 mantissa bits; the sign bit is 0).  Keys
// order like the values they truncate.  The per-coordinate rule
// compares thresholds instead of forming products: a -> RN32(a * inv_k) is
// non-decreasing for inv_k > 0, so RN32(a * inv_k) <= s_0 holds exactly for
// a <= T_k, the largest binary32 that passes; k_index_prep finds T_k once
// per call (a few ulp steps from s_0 / inv_k).  A key below T_k's key means a < T_k, a
// key above it a > T_k; only a key equal to T_k's leaves the comparison open,
// and then the coordinate's rows are read again for its exact maximum (at
// the scales used here, about one coordinate in ten thousand).  The count
// #{k : a <= T_k} needs no loop over k when no binade holds two thresholds
// (scales at least about twice apart, as 16^k): every T_k in a higher binade
// than a's counts, none in a lower one, so a table over the 256 values of the
// exponent field gives the count above a's binade and the key of the one
// threshold inside it, and a coordinate costs one lookup and two compares.
// Otherwise the block compares each key with the K thresholds' keys.  The
// thresholds, their keys and the table are formed once per call
// (k_index_prep) rather than in each of the pass's blocks: at 2^30
// coordinates that prologue was most of the pass's VALU work.
constexpr int kIndexOcts = 4;
constexpr int64_t kIndexTile = kIndexOcts * kBlock;
static_assert(kBlock == 256, "the exponent table has one entry per thread");

// Largest binary32 a >= 0 with RN32(a * inv) <= s0, for 0 < inv; 0 when inv
// is infinite (then no positive a passes).
__device__ float index_threshold(float inv, float s0)
{
    if (!(inv <= kFloatMax))
        return 0.0f;
    const double q = static_cast<double>(s0) / static_cast<double>(inv);
    float a = q >= static_cast<double>(kFloatMax) ? kFloatMax : static_cast<float>(q);
    // RN32(q) is within an ulp or two of the boundary; the loops are bounded
    // for safety and take at most a few steps
    for (int i = 0; i < 64 && a > 0.0f && a * inv > s0; ++i)
        a = __builtin_bit_cast(float, __builtin_bit_cast(uint32_t, a) - 1u);
    for (int i = 0; i < 64 && a < kFloatMax; ++i) {
        const float n = __builtin_bit_cast(float, __builtin_bit_cast(uint32_t, a) + 1u);
        if (!(n * inv <= s0))
            break;
        a = n;
    }
    return a;
}

// Scale index of amax from the thresholds: #{k < K : amax <= T_k} - 1 (the
// rule of index_of), K - 1 for a zero amax or on the zero path.
__device__ __forceinline__ uint32_t index_from_count(float amax, int32_t count, int32_t K, bool zero)
{
    if (zero || !(amax > 0.0f))
        return static_cast<uint32_t>(K - 1);
    return static_cast<uint32_t>(count > 0 ? count - 1 : 0);
}

// The index of coordinate i from its exact maximum over the rows (the value
// whose key the norm pass kept); M <= kFuseRows.  Rows past M re-read row
// M - 1 (no change to the maximum), so that the loads carry no branch and
// all are in flight at once.
__device__ __forceinline__ uint32_t index_exact(const float* __restrict__ g, int64_t ldg, int32_t M, int64_t i,
                                             const float* thr, int32_t K)
{
    float v[kFuseRows];
#pragma unroll
    for (int m = 0; m < kFuseRows; ++m)
        v[m] = g[static_cast<int64_t>(m < M ? m : M - 1) * ldg + i];
    float a = 0.0f;
#pragma unroll
    for (int m = 0; m < kFuseRows; ++m)
        a = fmaxf(a, usable_or_zero(v[m]));
    int32_t count = 0;
    for (int k = 0; k < K; ++k)
        count += a <= thr[k] ? 1 : 0;
    return index_from_count(a, count, K, false);
}

// Index of the coordinate with key `key` from the exponent table (entry e:
// the index when the key is not below the limit key of binade e, and that
// key; binades without a threshold hold 0x10000, which every key is below,
// with their index lowered by one); `tie` collects a key equal to the limit's.
__device__ __forceinline__ uint32_t index_from_key(const uint2* tab, uint32_t key, bool& tie)
{
    const uint2 t = tab[key >> 8];
    tie |= key == t.y;
    return t.x + (key < t.y ? 1u : 0u);
}

// The same from the K thresholds' keys (binades that hold two thresholds).
__device__ __forceinline__ uint32_t index_from_keys(const uint32_t* hk, int32_t K, uint32_t key, bool& tie)
{
    int32_t count = 0;
    for (int k = 0; k < K; ++k) {
        count += key < hk[k] ? 1 : 0;
        tie |= key == hk[k];
    }
    return static_cast<uint32_t>(count > 0 ? count - 1 : 0);
}

// Key c of an octet's eight (two per 32-bit word, the lower coordinate in
// the low half).
__device__ __forceinline__ uint32_t octet_key(const u32x4& kv, int c)
{
    const uint32_t w = c < 2 ? kv.x : c < 4 ? kv.y : c < 6 ? kv.z : kv.w;
    return (c & 1) ? w >> 16 : w & 0xFFFFu;
}

// One block: the rows' sums S_m from their kRowsumSpan-partial sums (the
// order of k_rowsum), W = RN32(sqrt(max_m S_m)) (NaN if any S_m is NaN, as
// k_finish), stored to *wptr, then the index pass's constants for the call:
// thresholds T_k, their keys and the exponent table (thread e forms entry e:
// the thresholds in higher binades, every key of binade e being below
// theirs, and the one inside binade e).  On the zero path every coordinate
// gets K - 1.
__global__ __launch_bounds__(kBlock) void k_index_prep(const double* __restrict__ sub, int64_t nsub, int32_t M,
                                                       double* __restrict__ rows, float* __restrict__ wptr,
                                                       ScaleSet S, IndexTables* __restrict__ T)
{
    __shared__ double wave_part[kBlock / 64];
    __shared__ double row_part[kFuseRows][kBlock / 64];
    __shared__ double row_s[kFuseRows];
    __shared__ float thr_s[kMaxScales];
    __shared__ uint32_t hk_s[kMaxScales];
    __shared__ float w_s;
    if (nsub <= kBlock) {
        // at most one partial per thread and row (every d below 2^32): all
        // rows' loads at once, then for each row the arithmetic of
        // rowsum_span (its sequential sum is the one value plus zeros,
        // exactly that value; then the butterfly and the four waves in order)
        const int lane = threadIdx.x & 63;
        const int wave = threadIdx.x >> 6;
        double x[kFuseRows];
#pragma unroll
        for (int m = 0; m < kFuseRows; ++m)
            x[m] = 0.0 + (m < M && threadIdx.x < nsub ? sub[static_cast<int64_t>(m) * nsub + threadIdx.x] : 0.0);
#pragma unroll
        for (int m = 0; m < kFuseRows; ++m) {
            const double s = wave_sum(x[m]);
            if (lane == 0)
                row_part[m][wave] = s;
        }
        __syncthreads();
        if (threadIdx.x < M) {
            const double* w4 = row_part[threadIdx.x];
            const double r = (w4[0] + w4[1]) + (w4[2] + w4[3]);
            rows[threadIdx.x] = r;
            row_s[threadIdx.x] = r;
        }
    } else {
        for (int32_t m = 0; m < M; ++m) {
            const double r = rowsum_span(sub + static_cast<int64_t>(m) * nsub, 0, nsub, wave_part);
            if (threadIdx.x == 0) {
                rows[m] = r;
                row_s[m] = r;
            }
            __syncthreads();  // wave_part is written again by the next row
        }
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        double best = 0.0;
        bool any_nan = false;
        for (int32_t m = 0; m < M; ++m) {
            const double r = row_s[m];
            any_nan = any_nan || (r != r);
            best = r > best ? r : best;
        }
        const float W = any_nan ? __builtin_nanf("") : static_cast<float>(sqrt(best));
        *wptr = W;
        w_s = W;
    }
    __syncthreads();
    const float W = w_s;
    const float s0 = S.s[0];
    const int32_t K = S.K;
    const bool zero = zero_path(W, div_rn32(s0, W));
    if (threadIdx.x < K) {
        const float t = zero ? 0.0f : index_threshold(div_rn32(S.s[threadIdx.x], W), s0);
        thr_s[threadIdx.x] = t;
        hk_s[threadIdx.x] = __builtin_bit_cast(uint32_t, t) >> 15;
        T->thr[threadIdx.x] = t;
        T->hk[threadIdx.x] = __builtin_bit_cast(uint32_t, t) >> 15;
    }
    __syncthreads();
    int crowded = 0;
    {
        const uint32_t e = threadIdx.x;
        int32_t above = 0, inside = 0;
        uint32_t kin = 0u;
        for (int k = 0; k < K; ++k) {
            const uint32_t be = __builtin_bit_cast(uint32_t, thr_s[k]) >> 23;
            above += be > e ? 1 : 0;
            if (be == e) {
                ++inside;
                kin = hk_s[k];
            }
        }
        uint2 ent;
        if (zero) {
            ent.x = static_cast<uint32_t>(K - 2);
            ent.y = 0x10000u;
        } else {
            // #{k : a <= T_k} - 1 = above - 1 + [key below kin]; with nothing
            // above, index 0 either way (nor does a tie matter then)
            crowded = inside > 1 ? 1 : 0;
            const bool limit = inside > 0 && above > 0;
            ent.x = static_cast<uint32_t>(above > 0 ? above - 1 : 0) - (limit ? 0u : 1u);
            ent.y = limit ? kin : 0x10000u;
        }
        T->tab[e] = ent;
    }
    const bool by_table = __syncthreads_or(crowded) == 0;
    if (threadIdx.x == 0)
        T->by_table = by_table ? 1 : 0;
}

// NIB: the index stored as 4-bit fields (an octet's eight in one 32-bit
// store), as in k_index.
template <bool NT, bool NIB>
__global__ __launch_bounds__(kBlock) void k_index_max(const uint16_t* __restrict__ keys,
                                                      const float* __restrict__ g, int64_t ldg, int64_t d,
                                                      int32_t M, const IndexTables* __restrict__ T, int32_t K,
                                                      uint8_t* __restrict__ idx)
{
    __shared__ float thr_s[kMaxScales];
    __shared__ uint32_t hk_s[kMaxScales];
    __shared__ uint2 tab_s[256];
    const int64_t noct = d >> 3;
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kIndexTile;
    const int64_t tile0 = static_cast<int64_t>(blockIdx.x) * kIndexTile;
    u32x4 kv[kIndexOcts];
#pragma unroll
    for (int j = 0; j < kIndexOcts; ++j) {
        const int64_t o = tile0 + threadIdx.x + kBlock * j;
        kv[j] = o < noct ? load_nt(reinterpret_cast<const uint32_t*>(keys + (o << 3))) : u32x4{0u, 0u, 0u, 0u};
    }
    // the call's constants (k_index_prep), through LDS
    tab_s[threadIdx.x] = T->tab[threadIdx.x];
    if (threadIdx.x < K) {
        thr_s[threadIdx.x] = T->thr[threadIdx.x];
        hk_s[threadIdx.x] = T->hk[threadIdx.x];
    }
    const bool by_table = T->by_table != 0;
    __syncthreads();

    for (int64_t t0 = tile0; t0 < noct; t0 += stride) {
        if (t0 != tile0) {
#pragma unroll
            for (int j = 0; j < kIndexOcts; ++j) {
                const int64_t o = t0 + threadIdx.x + kBlock * j;
                kv[j] = o < noct ? load_nt(reinterpret_cast<const uint32_t*>(keys + (o << 3)))
                                 : u32x4{0u, 0u, 0u, 0u};
            }
        }
        uint32_t ties = 0u;  // octets j holding a key equal to a threshold's
        if (by_table) {
#pragma unroll
            for (int j = 0; j < kIndexOcts; ++j) {
                const int64_t o = t0 + threadIdx.x + kBlock * j;
                if (o >= noct)
                    continue;
                const uint32_t k8[8] = {kv[j].x & 0xFFFFu, kv[j].x >> 16, kv[j].y & 0xFFFFu, kv[j].y >> 16,
                                        kv[j].z & 0xFFFFu, kv[j].z >> 16, kv[j].w & 0xFFFFu, kv[j].w >> 16};
                uint32_t ix[8];
                bool tie = false;
#pragma unroll
                for (int c = 0; c < 8; ++c)
                    ix[c] = index_from_key(tab_s, k8[c], tie);
                if (NIB) {
                    const uint32_t packed = ix[0] | (ix[1] << 4) | (ix[2] << 8) | (ix[3] << 12) | (ix[4] << 16) |
                                            (ix[5] << 20) | (ix[6] << 24) | (ix[7] << 28);
                    if (NT)
                        __builtin_nontemporal_store(packed, reinterpret_cast<uint32_t*>(idx + (o << 2)));
                    else
                        *reinterpret_cast<uint32_t*>(idx + (o << 2)) = packed;
                } else {
                    u32x2 packed;
                    packed.x = ix[0] | (ix[1] << 8) | (ix[2] << 16) | (ix[3] << 24);
                    packed.y = ix[4] | (ix[5] << 8) | (ix[6] << 16) | (ix[7] << 24);
                    if (NT)
                        __builtin_nontemporal_store(packed, reinterpret_cast<u32x2*>(idx + (o << 3)));
                    else
                        *reinterpret_cast<u32x2*>(idx + (o << 3)) = packed;
                }
                ties |= tie ? 1u << j : 0u;
            }
        } else {
            // binades holding two thresholds (unusual scale sets): the keys
            // again from memory, one octet at a time
#pragma unroll 1
            for (int j = 0; j < kIndexOcts; ++j) {
                const int64_t o = t0 + threadIdx.x + kBlock * j;
                if (o >= noct)
                    continue;
                const u32x4 kj = load_nt(reinterpret_cast<const uint32_t*>(keys + (o << 3)));
                u32x2 packed = {0u, 0u};
                bool tie = false;
#pragma unroll 1
                for (int c = 0; c < 8; ++c) {
                    const uint32_t v = index_from_keys(hk_s, K, octet_key(kj, c), tie);
                    if (NIB)
                        packed.x |= v << (4 * c);
                    else if (c < 4)
                        packed.x |= v << (8 * c);
                    else
                        packed.y |= v << (8 * (c - 4));
                }
                if (NIB)
                    *reinterpret_cast<uint32_t*>(idx + (o << 2)) = packed.x;
                else
                    *reinterpret_cast<u32x2*>(idx + (o << 3)) = packed;
                ties |= tie ? 1u << j : 0u;
            }
        }
        // keys equal to a threshold's (rare): those coordinates' indices again
        // from their exact maxima, over the index bytes just stored
        while (ties != 0u) {
            const int j = __builtin_ctz(ties);
            ties &= ties - 1u;
            const int64_t o = t0 + threadIdx.x + kBlock * j;
            const u32x4 kj = load_nt(reinterpret_cast<const uint32_t*>(keys + (o << 3)));
            uint32_t word = 0u;  // NIB: the octet's eight fields, stored again whole
#pragma unroll 1
            for (int c = 0; c < 8; ++c) {
                bool tc = false;
                const uint32_t key = octet_key(kj, c);
                uint32_t v = by_table ? index_from_key(tab_s, key, tc) : index_from_keys(hk_s, K, key, tc);
                if (tc)
                    v = index_exact(g, ldg, M, (o << 3) + c, thr_s, K);
                if (NIB)
                    word |= v << (4 * c);
                else if (tc)
                    idx[(o << 3) + c] = static_cast<uint8_t>(v);
            }
            if (NIB)
                *reinterpret_cast<uint32_t*>(idx + (o << 2)) = word;
        }
    }
    // the d % 8 trailing coordinates: threads of block 0 (with 4-bit fields
    // thread 0 alone, since two coordinates share a byte)
    const int64_t t = (noct << 3) + threadIdx.x;
    if (blockIdx.x == 0 && t < d && (!NIB || threadIdx.x == 0)) {
        uint32_t nib = 0u;
        for (int64_t i = t; i < (NIB ? d : t + 1); ++i) {
            bool tie = false;
            const uint32_t key = keys[i];
            uint32_t v = by_table ? index_from_key(tab_s, key, tie) : index_from_keys(hk_s, K, key, tie);
            if (tie)
                v = index_exact(g, ldg, M, i, thr_s, K);
            if (!NIB) {
                idx[i] = static_cast<uint8_t>(v);
            } else {
                nib |= v << (4 * ((i - t) & 1));
                if (((i - t) & 1) || i + 1 == d) {
                    idx[i >> 1] = static_cast<uint8_t>(nib);
                    nib = 0u;
                }
            }
        }
    }
}
// ---------------------------------------------------------------------------
// Quantisation.  One thread handles a group of 8 consecutive coordinates,
// which is exactly one Philox block: its eight 16-bit halves are the high
// halves of the coordinates' uniform words (coordinate j < 4 takes the low
// half of word j, coordinate j >= 4 the high half of word j - 4).  The low
// halves (a second block with counter word 3 = 1) are drawn only when some
// coordinate's high half ties its threshold's (probability 2^-16 each).
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t half_of(const uint32_t w[4], int j)
{
    return j < 4 ? (w[j] & 0xFFFFu) : (w[j - 4] >> 16);
}

// Quantise the 8 coordinates v[] of group q of `worker`; returns the codes.
__device__ __forceinline__ void quantise_group(const float v[8], const float inv[8], float s0, uint64_t q,
                                               uint32_t worker, uint32_t key0, uint32_t key1, int32_t code[8])
{
    const uint4 hi = philox4x32_10(static_cast<uint32_t>(q), static_cast<uint32_t>(q >> 32), worker, 0u,
                                   key0, key1);
    const uint32_t hw[4] = {hi.x, hi.y, hi.z, hi.w};
    float x[8];
    bool tie[8];
    bool any_tie = false;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        code[j] = quantise_hi(v[j], inv[j], s0, half_of(hw, j), &tie[j], &x[j]);
        any_tie = any_tie || tie[j];
    }
    if (__builtin_expect(any_tie, 0)) {
        const uint4 lo = philox4x32_10(static_cast<uint32_t>(q), static_cast<uint32_t>(q >> 32), worker, 1u,
                                       key0, key1);
        const uint32_t lw[4] = {lo.x, lo.y, lo.z, lo.w};
#pragma unroll
        for (int j = 0; j < 8; ++j)
            if (tie[j])
                code[j] = quantise_tie(v[j], x[j], half_of(lw, j));
    }
}

// Wave tiles.  A wave quantises 512 consecutive coordinates (64 Philox blocks)
// with perfectly coalesced accesses: lane t holds coordinates 4t..4t+3 ("A")
// and 256+4t..256+4t+3 ("B") of the tile.  The A coordinates of lanes 2u and
// 2u+1 form block 64T+u, their B coordinates block 64T+32+u.  Even lane 2u
// computes block 64T+u, odd lane 2u+1 block 64T+32+u, and the pair swaps the
// 16-bit halves the other needs with one DPP move per word pair.
__device__ __forceinline__ uint32_t swap_pair(uint32_t x)
{
    return static_cast<uint32_t>(__builtin_amdgcn_mov_dpp(static_cast<int>(x), 0xB1, 0xF, 0xF, false));
}

// Halves of this lane's A and B coordinates from its own block's words w:
// a01/a23 pack coordinates A0..A3 (coordinate 2k in the low half), b01/b23
// likewise for B.  Even lanes keep the low halves of their own words (their
// A coordinates) and receive the partner's low halves (their B coordinates);
// odd lanes keep high halves (B) and receive the partner's high halves (A).
__device__ __forceinline__ void tile_halves(uint4 w, bool odd, uint32_t* a01, uint32_t* a23, uint32_t* b01,
                                            uint32_t* b23)
{
    const uint32_t sel_lo = 0x05040100u;  // low halves of (src1, src0)
    const uint32_t sel_hi = 0x07060302u;  // high halves of (src1, src0)
    const uint32_t sel_keep = odd ? sel_hi : sel_lo;
    const uint32_t sel_send = odd ? sel_lo : sel_hi;
    const uint32_t keep01 = __builtin_amdgcn_perm(w.y, w.x, sel_keep);
    const uint32_t keep23 = __builtin_amdgcn_perm(w.w, w.z, sel_keep);
    const uint32_t recv01 = swap_pair(__builtin_amdgcn_perm(w.y, w.x, sel_send));
    const uint32_t recv23 = swap_pair(__builtin_amdgcn_perm(w.w, w.z, sel_send));
    *a01 = odd ? recv01 : keep01;
    *a23 = odd ? recv23 : keep23;
    *b01 = odd ? keep01 : recv01;
    *b23 = odd ? keep23 : recv23;
}

__device__ __forceinline__ uint32_t half16(uint32_t packed01, uint32_t packed23, int j)
{
    const uint32_t w = j < 2 ? packed01 : packed23;
    return (j & 1) ? (w >> 16) : (w & 0xFFFFu);
}

// BITS = 8: int8 codes.  BITS = 4 or 2: codes packed low bits first, two or
// four to a byte (every |code| <= s_0 fits the field; checked on the host).
template <int BITS>
__device__ __forceinline__ uint32_t pack_field(const int32_t c[4])
{
    constexpr uint32_t mask = (1u << BITS) - 1u;
    uint32_t w = 0u;
#pragma unroll
    for (int j = 0; j < 4; ++j)
        w |= (static_cast<uint32_t>(c[j]) & mask) << (BITS * j);
    return w;
}

// Stores four consecutive codes held as 16-bit lanes of p01 (codes 0, 1) and
// p23 (codes 2, 3) at coordinate `coord` of a code row.
template <int BITS, bool NT>
__device__ __forceinline__ void store_pairs(uint8_t* row, int64_t coord, uint32_t p01, uint32_t p23)
{
    // the low byte of each lane: codes 0..3 in bytes 0..3
    const uint32_t w = __builtin_amdgcn_perm(p23, p01, 0x06040200u);
    if (BITS == 8) {
        uint32_t* p = reinterpret_cast<uint32_t*>(row + coord);
        if (NT)
            __builtin_nontemporal_store(w, p);
        else
            *p = w;
    } else if (BITS == 4) {
        const uint32_t x = w & 0x0F0F0F0Fu;
        const uint32_t y = x | (x >> 4);  // byte 0: codes 0, 1; byte 2: codes 2, 3
        const uint16_t v = static_cast<uint16_t>(__builtin_amdgcn_perm(0u, y, 0x0C0C0200u));
        uint16_t* p = reinterpret_cast<uint16_t*>(row + coord / 2);
        if (NT)
            __builtin_nontemporal_store(v, p);
        else
            *p = v;
    } else {
        const uint32_t x = w & 0x03030303u;
        const uint32_t y = x | (x >> 6);  // byte 0: codes 0, 1; byte 2: codes 2, 3
        const uint8_t v = static_cast<uint8_t>(y | (y >> 12));
        if (NT)
            __builtin_nontemporal_store(v, row + coord / 4);
        else
            row[coord / 4] = v;
    }
}

// Replaces 16-bit lane (j & 1) of *p with code c.
__device__ __forceinline__ void set_lane16(uint32_t* p, int j, int32_t c)
{
    const uint32_t u = static_cast<uint32_t>(c) & 0xFFFFu;
    *p = (j & 1) ? ((*p & 0xFFFFu) | (u << 16)) : ((*p & 0xFFFF0000u) | u);
}

// One tile's inputs for one lane: its A and B gradient quads and, with
// several scales, their four scale indices each.
struct TileIn {
    f32x4 A, B;
    uint32_t ka, kb;
};

// The four 4-bit index fields of a 16-bit word (coordinate 2j in the low
// nibble of byte j) spread to the four bytes of a word, the byte layout.
__device__ __forceinline__ uint32_t nibbles_to_bytes(uint32_t h)
{
    return (h & 0xFu) | ((h << 4) & 0xF00u) | ((h << 8) & 0xF0000u) | ((h << 12) & 0xF000000u);
}

// Index k*_i of the 4-bit layout: the low nibble of byte i / 2 for even i,
// the high nibble for odd i.
__device__ __forceinline__ uint32_t nibble_at(const uint8_t* __restrict__ idx4, int64_t i)
{
    return (static_cast<uint32_t>(idx4[i >> 1]) >> ((i & 1) * 4)) & 0xFu;
}

// NIB: the index is held as 4-bit fields (two coordinates a byte); its
// fields are spread to bytes here, so that everything after the load is the
// byte layout's.
template <bool MULTI, bool NIB = false>
__device__ __forceinline__ TileIn load_tile(const float* __restrict__ row, const uint8_t* __restrict__ idx,
                                            int64_t a_off)
{
    TileIn in;
    in.A = load_nt(row + a_off);
    in.B = load_nt(row + a_off + 256);
    if (MULTI && NIB) {
        in.ka = nibbles_to_bytes(*reinterpret_cast<const uint16_t*>(idx + (a_off >> 1)));
        in.kb = nibbles_to_bytes(*reinterpret_cast<const uint16_t*>(idx + ((a_off + 256) >> 1)));
    } else {
        in.ka = MULTI ? *reinterpret_cast<const uint32_t*>(idx + a_off) : 0u;
        in.kb = MULTI ? *reinterpret_cast<const uint32_t*>(idx + a_off + 256) : 0u;
    }
    return in;
}

// The eight codes of one lane for tile T of worker `worker`, as four 16-bit
// lane pairs (A0 A1, A2 A3, B0 B1, B2 B3).  v: the lane's coordinates;
// inv: their s_k / W, times 2^16 when PRE (then s0x = s0 * 2^16).  Every lane
// of the wave must call it (DPP exchange, wave-uniform branches).
template <bool PRE>
__device__ __forceinline__ void tile_codes(const float v[8], const float inv[8], float s0x, int64_t T,
                                           uint32_t worker, uint32_t key0, uint32_t key1, uint32_t one2,
                                           uint32_t p[4])
{
    const int lane = threadIdx.x & 63;
    const bool odd = (lane & 1) != 0;
    const uint64_t q = static_cast<uint64_t>(T << 6) + static_cast<uint64_t>(lane >> 1) + (odd ? 32u : 0u);
    uint32_t a01, a23, b01, b23;
    tile_halves(philox4x32_10(static_cast<uint32_t>(q), static_cast<uint32_t>(q >> 32), worker, 0u, key0, key1),
                odd, &a01, &a23, &b01, &b23);
    float xs[8];
    if (PRE) {
        // every table entry is finite, so |v| * inv is NaN or infinite only
        // for NaN or infinite v, which quantise to 0 (wave-uniform, rare)
        bool bad = false;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            xs[j] = fminf(fabsf(v[j]) * inv[j], s0x);
            bad = bad || __builtin_amdgcn_classf(v[j], kNonFinite);
        }
        if (__builtin_expect(__ballot(bad) != 0, 0)) {
#pragma unroll
            for (int j = 0; j < 8; ++j)
                xs[j] = __builtin_amdgcn_classf(v[j], kNonFinite) ? 0.0f : xs[j];
        }
    } else {
        // entries may be infinite (0 * inf is NaN): select by class
#pragma unroll
        for (int j = 0; j < 8; ++j)
            xs[j] = scaled_magnitude(v[j], inv[j], s0x) * 65536.0f;
    }
    uint32_t Tw[8];
    bool tie[8];
    bool any_tie = false;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        Tw[j] = static_cast<uint32_t>(xs[j]);
        const uint32_t h = j < 4 ? half16(a01, a23, j) : half16(b01, b23, j - 4);
        tie[j] = (Tw[j] & 0xFFFFu) == h;
        any_tie = any_tie || tie[j];
    }
    p[0] = pair_codes(Tw[0], Tw[1], v[0], v[1], a01, one2);
    p[1] = pair_codes(Tw[2], Tw[3], v[2], v[3], a23, one2);
    p[2] = pair_codes(Tw[4], Tw[5], v[4], v[5], b01, one2);
    p[3] = pair_codes(Tw[6], Tw[7], v[6], v[7], b23, one2);
    // wave-uniform branch (the DPP exchange needs every lane): draw the low
    // halves from the purpose-1 blocks when any lane has a tie
    if (__builtin_expect(__ballot(any_tie) != 0, 0)) {
        tile_halves(philox4x32_10(static_cast<uint32_t>(q), static_cast<uint32_t>(q >> 32), worker, 1u, key0, key1),
                    odd, &a01, &a23, &b01, &b23);
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const uint32_t h = j < 4 ? half16(a01, a23, j) : half16(b01, b23, j - 4);
            if (tie[j])
                set_lane16(&p[j >> 1], j, quantise_tie_scaled(v[j], xs[j], Tw[j], h));
        }
    }
}

// One tile of one code row: the codes from the lane's loaded inputs, then
// the stores.  inv_t / inv0 hold s_k / W, multiplied by 2^16 when PRE (then
// s0x = s0 * 2^16 too), so that xs = x * 2^16 comes out of one multiply and
// one min; without PRE (an entry is above 2^100, or infinite) the 2^16 is
// applied after the min.  Both give xs = RN(|v| s_k / W) * 2^16 exactly
// whenever |v| s_k / W is a normal number, and T = floor(xs) = 0 with a zero
// threshold low half otherwise, so the codes do not depend on PRE.
template <bool MULTI, int BITS, bool PRE, bool NT>
__device__ __forceinline__ void code_tile(const TileIn& in, uint8_t* __restrict__ out, int64_t T,
                                          const float* inv_t, float inv0, float s0x, uint32_t kmax,
                                          uint32_t worker, uint32_t key0, uint32_t key1, uint32_t one2)
{
    const float v[8] = {in.A.x, in.A.y, in.A.z, in.A.w, in.B.x, in.B.y, in.B.z, in.B.w};
    float inv[8];
    if (MULTI) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            inv[j] = inv_t[min((in.ka >> (8 * j)) & 0xFFu, kmax)];
            inv[j + 4] = inv_t[min((in.kb >> (8 * j)) & 0xFFu, kmax)];
        }
    } else {
#pragma unroll
        for (int j = 0; j < 8; ++j)
            inv[j] = inv0;
    }
    uint32_t p[4];
    tile_codes<PRE>(v, inv, s0x, T, worker, key0, key1, one2, p);
    const int64_t a_off = (T << 9) + 4 * (threadIdx.x & 63);
    store_pairs<BITS, NT>(out, a_off, p[0], p[1]);
    store_pairs<BITS, NT>(out, a_off + 256, p[2], p[3]);
}

// The whole tiles of one code row when the grid covers them all at once: the
// wave's tile `first` and, with several scales and tpw = 2, first + 1, as
// straight-line code.  With one scale (tpw = 1) the tile arrives already
// loaded in `in0`.  The loop form below, run with the same tiles, measured
// 9% slower with one scale and 1% slower with several (its 64-bit tile
// bounds are compared on the vector unit).
template <bool MULTI, int BITS, bool PRE, bool NT>
__device__ __forceinline__ void quantise_few(const float* __restrict__ row, uint8_t* __restrict__ out,
                                             const uint8_t* __restrict__ idx, int64_t ntiles, int64_t first,
                                             int32_t tpw, const TileIn& in0, const float* inv_t, float inv0,
                                             float s0x, uint32_t kmax, uint32_t worker, uint32_t key0,
                                             uint32_t key1)
{
    uint32_t one2 = 0x00010001u;
    asm("" : "+s"(one2));
    const int lane = threadIdx.x & 63;
    if (first < ntiles) {
        const TileIn in = MULTI ? load_tile<MULTI>(row, idx, (first << 9) + 4 * lane) : in0;
        code_tile<MULTI, BITS, PRE, NT>(in, out, first, inv_t, inv0, s0x, kmax, worker, key0, key1, one2);
    }
    if (MULTI && tpw == 2 && first + 1 < ntiles) {
        const TileIn in = load_tile<MULTI>(row, idx, ((first + 1) << 9) + 4 * lane);
        code_tile<MULTI, BITS, PRE, NT>(in, out, first + 1, inv_t, inv0, s0x, kmax, worker, key0, key1, one2);
    }
}

// The whole tiles of one code row on a capped grid: each wave takes `tpw`
// consecutive tiles from `first`, then strides by the grid.
template <bool MULTI, int BITS, bool PRE, bool NT>
__device__ __forceinline__ void quantise_tiles(const float* __restrict__ row, uint8_t* __restrict__ out,
                                               const uint8_t* __restrict__ idx, int64_t ntiles, int64_t first,
                                               int64_t stride, const TileIn& in0, const float* inv_t, float inv0,
                                               float s0x, uint32_t kmax, uint32_t worker, uint32_t key0,
                                               uint32_t key1, int32_t tpw)
{
    const int lane = threadIdx.x & 63;
    uint32_t one2 = 0x00010001u;
    asm("" : "+s"(one2));
    for (int64_t c0 = first; c0 < ntiles; c0 += stride) {
        const int64_t c1 = c0 + tpw < ntiles ? c0 + tpw : ntiles;
        for (int64_t T = c0; T < c1; ++T) {
            const TileIn in = (!MULTI && T == first) ? in0 : load_tile<MULTI>(row, idx, (T << 9) + 4 * lane);
            code_tile<MULTI, BITS, PRE, NT>(in, out, T, inv_t, inv0, s0x, kmax, worker, key0, key1, one2);
        }
    }
}

// The coordinates of one row past its last whole tile (fewer than 512), in
// groups of 8 contiguous coordinates, one per lane of one wave.  inv_s holds
// s_k / W (not scaled).
template <bool MULTI, int BITS>
__device__ __forceinline__ void quantise_tail(const float* __restrict__ row, uint8_t* __restrict__ out,
                                              const uint8_t* __restrict__ idx, int64_t d, int64_t ntiles,
                                              const float* inv_s, float inv0, float s0, uint32_t kmax,
                                              uint32_t worker, uint32_t key0, uint32_t key1)
{
    const int64_t q = (ntiles << 6) + (threadIdx.x & 63);
    const int64_t base = q << 3;
    if (base >= d)
        return;
    float v[8], inv[8];
    int32_t code[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const bool in = base + j < d;
        v[j] = in ? row[base + j] : 0.0f;
        inv[j] = MULTI ? inv_s[min(static_cast<uint32_t>(in ? idx[base + j] : 0), kmax)] : inv0;
    }
    quantise_group(v, inv, s0, static_cast<uint64_t>(q), worker, key0, key1, code);
    if (BITS == 8) {
#pragma unroll
        for (int j = 0; j < 8; ++j)
            if (base + j < d)
                out[base + j] = static_cast<uint8_t>(code[j]);
    } else {
        // the group's 8 codes fill whole bytes of its own (coordinates past d
        // have code 0); the packed row holds them
        if (BITS == 4)
            *reinterpret_cast<uint32_t*>(out + base / 2) = pack_field<4>(code) | (pack_field<4>(code + 4) << 16);
        else
            *reinterpret_cast<uint16_t*>(out + base / 4) =
                static_cast<uint16_t>(pack_field<2>(code) | (pack_field<2>(code + 4) << 8));
    }
}

// The quantiser: MULTI with a per-coordinate scale index, BITS the code
// width (8, or 4 / 2 packed), NT codes stored nontemporally (the launcher sets
// it for launches that write more than kCodesNontemporalBytes).
template <bool MULTI, int BITS, bool NT>
__global__ __launch_bounds__(kBlock) void k_quantise(const float* __restrict__ g, int64_t d, int64_t ldg,
                                                     int32_t worker0, const float* __restrict__ wptr,
                                                     ScaleSet S, const uint8_t* __restrict__ idx,
                                                     uint32_t key0, uint32_t key1,
                                                     uint8_t* __restrict__ codes, int64_t ldc, int32_t tpw)
{
    __shared__ float inv_s[kMaxScales];   // s_k / W
    __shared__ float inv_p[kMaxScales];   // s_k / W * 2^16 when pre

    // 2-D grid: tile blocks in x, worker rows in y; each wave takes `tpw`
    // consecutive tiles (on a one-shot grid, only those), then strides by
    // the grid
    const int32_t r = blockIdx.y;
    const uint32_t worker = static_cast<uint32_t>(worker0) + static_cast<uint32_t>(r);
    const float* row = g + static_cast<int64_t>(r) * ldg;
    uint8_t* out = codes + static_cast<int64_t>(r) * ldc;
    const int64_t ntiles = d >> 9;
    const int32_t wave_in_block = __builtin_amdgcn_readfirstlane(static_cast<int32_t>(threadIdx.x >> 6));
    const int64_t first = (static_cast<int64_t>(blockIdx.x) * (kBlock / 64) + wave_in_block) * tpw;
    const int64_t stride = static_cast<int64_t>(gridDim.x) * (kBlock / 64) * tpw;

    // with one scale the first tile's loads go out before the tables are
    // formed, so that their latency covers the load of W and the division
    // (with several scales this measured slower, so there they stay in the
    // tile loop)
    TileIn in0 = {};
    if (!MULTI && first < ntiles)
        in0 = load_tile<MULTI>(row, idx, (first << 9) + 4 * (threadIdx.x & 63));

    const float W = *wptr;
    // tables; on the zero path every entry is 0, which makes every code 0
    const float q0 = div_rn32(S.s[0], W);
    const bool zero = zero_path(W, q0);
    // the largest entry is the last scale's; 2^16 times it stays finite
    const bool pre = zero || (MULTI ? div_rn32(S.s_last, W) : q0) <= 0x1p100f;
    float inv0 = 0.0f;
    if (MULTI) {
        if (threadIdx.x < S.K) {
            const float inv = zero ? 0.0f : div_rn32(S.s[threadIdx.x], W);
            inv_s[threadIdx.x] = inv;
            inv_p[threadIdx.x] = pre ? inv * 65536.0f : inv;
        }
        __syncthreads();
    } else {
        inv0 = zero ? 0.0f : q0;
    }
    const float s0 = S.s[0];
    const uint32_t kmax = static_cast<uint32_t>(S.K - 1);

    if (stride >= ntiles && tpw <= (MULTI ? 2 : 1)) {
        if (pre)
            quantise_few<MULTI, BITS, true, NT>(row, out, idx, ntiles, first, tpw, in0, inv_p, inv0 * 65536.0f,
                                                s0 * 65536.0f, kmax, worker, key0, key1);
        else
            quantise_few<MULTI, BITS, false, NT>(row, out, idx, ntiles, first, tpw, in0, inv_p, inv0, s0, kmax,
                                                 worker, key0, key1);
    } else if (pre)
        quantise_tiles<MULTI, BITS, true, NT>(row, out, idx, ntiles, first, stride, in0, inv_p, inv0 * 65536.0f,
                                              s0 * 65536.0f, kmax, worker, key0, key1, tpw);
    else
        quantise_tiles<MULTI, BITS, false, NT>(row, out, idx, ntiles, first, stride, in0, inv_p, inv0, s0, kmax,
                                               worker, key0, key1, tpw);

    // Coordinates past the last whole tile (fewer than 512): groups of 8
    // contiguous coordinates, one per lane of the first wave of block x = 0.
    if (blockIdx.x == 0 && threadIdx.x < 64)
        quantise_tail<MULTI, BITS>(row, out, idx, d, ntiles, inv_s, inv0, s0, kmax, worker, key0, key1);
}

// ---------------------------------------------------------------------------
// Integer sum of the rows' codes (the all-reduce), for int8 codes and for
// codes packed as 4- or 2-bit fields.  A block tile of 4096 coordinates:
// thread t unpacks coordinates 16t .. 16t+15 of the tile from one 16-, 8- or
// 4-byte load per row with signed bit-field extracts, eight rows' loads in
// flight at a time.  The tile's sums are then staged through LDS so that the
// int32 stores (and, when accumulating, the loads of the old sums) are
// coalesced: thread t writes quads t, t+256, t+512 and t+768 of the tile.
// With DEQ (1: one scale, 2: several) the same threads also apply the
// reconstruction to the sums they store, so that they need not be read again.
// ---------------------------------------------------------------------------
constexpr int64_t kSumTile = 4096;

// The reconstruction's inputs when it is fused into the sum.
struct DeqArgs {
    const float* w;
    const uint8_t* idx;  // [d] shared scale index (several scales)
    float* out;
    ScaleSet S;
    int32_t M;
    int32_t nt_sum;      // store the sums nontemporally (large d)
};

// The fused sum stores the int32 sums nontemporally when they exceed this
// many bytes: measured 2% faster steps at ResNet-50 and VGG-16 sizes (0.1 to
// 0.55 GB of sums), 1.7% slower at ResNet-18 size (45 MB).
constexpr int64_t kSumNontemporalBytes = int64_t(64) << 20;


// The 16 BITS-bit fields starting at p (16-byte aligned for BITS = 8, 8-byte
// for 4, 4-byte for 2).
template <int BITS>
__device__ __forceinline__ u32x4 load_fields(const uint8_t* p)
{
    u32x4 w = {0u, 0u, 0u, 0u};
    if (BITS == 8) {
        w = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
    } else if (BITS == 4) {
        const u32x2 h = __builtin_nontemporal_load(reinterpret_cast<const u32x2*>(p));
        w.x = h.x;
        w.y = h.y;
    } else {
        w.x = load_nt_u32(p);
    }
    return w;
}

template <int BITS>
__device__ __forceinline__ void add_fields(u32x4 w, int32_t acc[16])
{
#pragma unroll
    for (int j = 0; j < 16; ++j) {
        const int k = (j * BITS) / 32;
        const uint32_t word = k == 0 ? w.x : k == 1 ? w.y : k == 2 ? w.z : w.w;
        acc[j] += __builtin_amdgcn_sbfe(static_cast<int32_t>(word), (j * BITS) % 32, BITS);
    }
}

template <int BITS, int DEQ>
__global__ __launch_bounds__(kBlock) void k_sum(const uint8_t* __restrict__ codes, int64_t d, int32_t rows,
                                                int64_t ldc, int32_t accumulate, int32_t* __restrict__ sum,
                                                DeqArgs da)
{
    constexpr int kRowsInFlight = 8;
    // the tile's sums with one padding word after every 16, so that both the
    // row-of-16 writes and the quad reads are free of bank conflicts
    __shared__ int32_t stage[kSumTile + kSumTile / 16];
    __shared__ float deq_s[kMaxScales];
    const int t = threadIdx.x;
    if (DEQ) {
        // deq_k = RN32(W / (M s_k)) as in k_dequant; the barrier after the
        // first tile's staging publishes them
        const float W = *da.w;
        const bool zero = zero_path(W, div_rn32(da.S.s[0], W));
        if (t < da.S.K) {
            const float denom = static_cast<float>(static_cast<double>(da.M) * static_cast<double>(da.S.s[t]));
            deq_s[t] = zero ? 0.0f : div_rn32(W, denom);
        }
    }
    const int32_t kmax = da.S.K - 1;
    for (int64_t tile0 = static_cast<int64_t>(blockIdx.x) * kSumTile; tile0 < d;
         tile0 += static_cast<int64_t>(gridDim.x) * kSumTile) {
        // several scales: the index words of the thread's four quads
        uint32_t kq[4] = {0u, 0u, 0u, 0u};
        if (DEQ == 2) {
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const int64_t q0 = tile0 + 1024 * c + 4 * t;
                if (q0 + 4 <= d)
                    kq[c] = *reinterpret_cast<const uint32_t*>(da.idx + q0);
            }
        }
        const int64_t c0 = tile0 + 16 * t;
        int32_t acc[16];
#pragma unroll
        for (int j = 0; j < 16; ++j)
            acc[j] = 0;
        if (c0 < d) {
            // fields past d in the last group are read (they lie inside the
            // row's ldc bytes) and dropped below
            const uint8_t* p = codes + c0 * BITS / 8;
            int32_t r = 0;
            for (; r + kRowsInFlight <= rows; r += kRowsInFlight) {
                u32x4 w[kRowsInFlight];
#pragma unroll
                for (int u = 0; u < kRowsInFlight; ++u)
                    w[u] = load_fields<BITS>(p + static_cast<int64_t>(r + u) * ldc);
#pragma unroll
                for (int u = 0; u < kRowsInFlight; ++u)
                    add_fields<BITS>(w[u], acc);
            }
            for (; r < rows; ++r)
                add_fields<BITS>(load_fields<BITS>(p + static_cast<int64_t>(r) * ldc), acc);
        }
#pragma unroll
        for (int j = 0; j < 16; ++j)
            stage[17 * t + j] = acc[j];
        __syncthreads();
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const int L = 1024 * c + 4 * t;  // tile coordinate of the quad
            const int S = L + (L >> 4);      // its padded LDS index
            const int64_t q0 = tile0 + L;
            if (q0 + 4 <= d) {
                int4 a = make_int4(stage[S], stage[S + 1], stage[S + 2], stage[S + 3]);
                if (accumulate) {
                    const int4 o = *reinterpret_cast<const int4*>(sum + q0);
                    a.x += o.x; a.y += o.y; a.z += o.z; a.w += o.w;
                }
                if (DEQ && da.nt_sum)
                    __builtin_nontemporal_store(i32x4{a.x, a.y, a.z, a.w}, reinterpret_cast<i32x4*>(sum + q0));
                else
                    *reinterpret_cast<int4*>(sum + q0) = a;
                if (DEQ) {
                    f32x4 o;
                    if (DEQ == 2) {
                        const uint32_t kk = kq[c];
                        o.x = static_cast<float>(a.x) * deq_s[min(static_cast<int32_t>(kk & 0xFFu), kmax)];
                        o.y = static_cast<float>(a.y) * deq_s[min(static_cast<int32_t>((kk >> 8) & 0xFFu), kmax)];
                        o.z = static_cast<float>(a.z) * deq_s[min(static_cast<int32_t>((kk >> 16) & 0xFFu), kmax)];
                        o.w = static_cast<float>(a.w) * deq_s[min(static_cast<int32_t>(kk >> 24), kmax)];
                    } else {
                        const float f = deq_s[0];
                        o.x = static_cast<float>(a.x) * f;
                        o.y = static_cast<float>(a.y) * f;
                        o.z = static_cast<float>(a.z) * f;
                        o.w = static_cast<float>(a.w) * f;
                    }
                    store_nt(da.out + q0, o);
                }
            } else {
                for (int j = 0; j < 4 && q0 + j < d; ++j) {
                    const int32_t v = stage[S + j] + (accumulate ? sum[q0 + j] : 0);
                    sum[q0 + j] = v;
                    if (DEQ) {
                        const int32_t k = DEQ == 2 ? min(static_cast<int32_t>(da.idx[q0 + j]), kmax) : 0;
                        da.out[q0 + j] = static_cast<float>(v) * deq_s[k];
                    }
                }
            }
        }
        __syncthreads();  // the next tile reuses stage
    }
}

// ---------------------------------------------------------------------------
// Reconstruction: out_i = RN32(sum_i * deq_k), deq_k = RN32(W / (M s_k)).
// ---------------------------------------------------------------------------
template <bool MULTI>
__global__ __launch_bounds__(kBlock) void k_dequant(const int32_t* __restrict__ sum, int64_t d, int32_t M,
                                                    const float* __restrict__ wptr, ScaleSet S,
                                                    const uint8_t* __restrict__ idx, float* __restrict__ out)
{
    __shared__ float deq_s[kMaxScales];
    const int64_t nquad = d >> 2;
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock;
    const int64_t first = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
    // the first quad's loads go out before the tables are formed
    i32x4 s_first = {0, 0, 0, 0};
    uint32_t k_first = 0u;
    if (first < nquad) {
        s_first = load_nt(sum + (first << 2));
        if (MULTI)
            k_first = *reinterpret_cast<const uint32_t*>(idx + (first << 2));
    }

    const float W = *wptr;
    const float inv0 = div_rn32(S.s[0], W);
    const bool zero = zero_path(W, inv0);
    if (threadIdx.x < S.K) {
        // M * s_k is exactly representable in binary32 (checked on the host)
        const float denom = static_cast<float>(static_cast<double>(M) * static_cast<double>(S.s[threadIdx.x]));
        deq_s[threadIdx.x] = zero ? 0.0f : div_rn32(W, denom);
    }
    __syncthreads();
    const int32_t kmax = S.K - 1;
    const float deq0 = deq_s[0];

    for (int64_t q = first; q < nquad; q += stride) {
        i32x4 s;
        uint32_t kk = 0u;
        if (q == first) {
            s = s_first;
            kk = k_first;
        } else {
            s = load_nt(sum + (q << 2));
            if (MULTI)
                kk = *reinterpret_cast<const uint32_t*>(idx + (q << 2));
        }
        f32x4 o;
        if (MULTI) {
            const int32_t k0 = min(static_cast<int32_t>(kk & 0xFFu), kmax);
            const int32_t k1 = min(static_cast<int32_t>((kk >> 8) & 0xFFu), kmax);
            const int32_t k2 = min(static_cast<int32_t>((kk >> 16) & 0xFFu), kmax);
            const int32_t k3 = min(static_cast<int32_t>(kk >> 24), kmax);
            o.x = static_cast<float>(s.x) * deq_s[k0];
            o.y = static_cast<float>(s.y) * deq_s[k1];
            o.z = static_cast<float>(s.z) * deq_s[k2];
            o.w = static_cast<float>(s.w) * deq_s[k3];
        } else {
            o.x = static_cast<float>(s.x) * deq0;
            o.y = static_cast<float>(s.y) * deq0;
            o.z = static_cast<float>(s.z) * deq0;
            o.w = static_cast<float>(s.w) * deq0;
        }
        store_nt(out + (q << 2), o);
    }
    const int64_t t = (nquad << 2) + static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
    if (blockIdx.x == 0 && t < d) {
        int32_t k = 0;
        if (MULTI)
            k = min(static_cast<int32_t>(idx[t]), kmax);
        out[t] = static_cast<float>(sum[t]) * deq_s[k];
    }
}

// ---------------------------------------------------------------------------
// Quantise and sum in one pass (Eq. (8)/(12) and the all-reduce of Algorithm
// 1/2): the rows' codes, exactly those k_quantise would store, are added into
// the int32 sums in registers and never stored.  A wave takes one
// 512-coordinate tile (the lane layout of k_quantise: quads A = 4t .. 4t+3
// and B = 256+4t .. 256+4t+3) of every row in turn, so the shared index and
// the tables are looked up once per tile; the next row's loads go out before
// the current row is coded.  The tile's sums are then stored once (the old
// sums added first when accumulating) and, with DEQ, so is the reconstruction
// of those sums, RN32(sum * deq_k).  Per streamed row this moves 4 + 1 bytes
// in and 4 (+ 4 read when accumulating) per coordinate, against 6 + 9 for the
// quantiser followed by the sum.
// ---------------------------------------------------------------------------

// The codes of up to kPairRows rows are summed in the 16-bit lanes of the
// pair registers (|sum| <= 256 * 127 < 2^15, so the wrapped 16-bit sums are
// exact), then widened to int32.
constexpr int32_t kPairRows = 256;

template <bool NT>
__device__ __forceinline__ i32x4 load_sum4(const int32_t* p)
{
    if (NT)
        return __builtin_nontemporal_load(reinterpret_cast<const i32x4*>(p));
    return *reinterpret_cast<const i32x4*>(p);
}

template <bool NT>
__device__ __forceinline__ void store_sum4(int32_t* p, i32x4 v)
{
    if (NT)
        __builtin_nontemporal_store(v, reinterpret_cast<i32x4*>(p));
    else
        *reinterpret_cast<i32x4*>(p) = v;
}

// Adds the 16-bit lane sums of h[4] (codes A0 A1, A2 A3, B0 B1, B2 B3) to the
// int32 sums acc[8] and clears h.
__device__ __forceinline__ void widen_pairs(uint32_t h[4], int32_t acc[8])
{
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        acc[2 * j] += __builtin_amdgcn_sbfe(static_cast<int32_t>(h[j]), 0, 16);
        acc[2 * j + 1] += __builtin_amdgcn_sbfe(static_cast<int32_t>(h[j]), 16, 16);
        h[j] = 0u;
    }
}

// One tile of every row: `in` holds row 0's quads and the tile's index words,
// oldA / oldB the sums already stored (when ACC).  inv_t / inv0 / s0x as for
// code_tile.
template <bool MULTI, bool PRE, bool ACC, bool DEQ, bool NT, bool ROW1>
__device__ __forceinline__ void quant_sum_tile(const float* __restrict__ g, int64_t ldg, int32_t rows,
                                               uint32_t worker0, int64_t T, TileIn in, i32x4 oldA, i32x4 oldB,
                                               const float* inv_t, float inv0, float s0x, uint32_t kmax,
                                               uint32_t key0, uint32_t key1, uint32_t one2,
                                               int32_t* __restrict__ sum, const float* deq_t,
                                               float* __restrict__ out)
{
    const int lane = threadIdx.x & 63;
    const int64_t a_off = (T << 9) + 4 * lane;
    float inv[8];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        inv[j] = MULTI ? inv_t[min((in.ka >> (8 * j)) & 0xFFu, kmax)] : inv0;
        inv[j + 4] = MULTI ? inv_t[min((in.kb >> (8 * j)) & 0xFFu, kmax)] : inv0;
    }
    int32_t acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    uint32_t h[4] = {0u, 0u, 0u, 0u};
    int32_t pending = 0;
    f32x4 A = in.A, B = in.B;
    const int32_t nrows = ROW1 ? 1 : rows;
    for (int32_t r = 0; r < nrows; ++r) {
        f32x4 nA = A, nB = B;
        if (!ROW1 && r + 1 < nrows) {
            const float* nrow = g + static_cast<int64_t>(r + 1) * ldg;
            nA = load_nt(nrow + a_off);
            nB = load_nt(nrow + a_off + 256);
        }
        const float v[8] = {A.x, A.y, A.z, A.w, B.x, B.y, B.z, B.w};
        uint32_t p[4];
        tile_codes<PRE>(v, inv, s0x, T, worker0 + static_cast<uint32_t>(r), key0, key1, one2, p);
#pragma unroll
        for (int j = 0; j < 4; ++j)
            h[j] = __builtin_bit_cast(uint32_t, __builtin_bit_cast(u16x2, h[j]) + __builtin_bit_cast(u16x2, p[j]));
        if (++pending == kPairRows) {
            widen_pairs(h, acc);
            pending = 0;
        }
        A = nA;
        B = nB;
    }
    widen_pairs(h, acc);
    i32x4 sa = {acc[0], acc[1], acc[2], acc[3]};
    i32x4 sb = {acc[4], acc[5], acc[6], acc[7]};
    if (ACC) {
        sa += oldA;
        sb += oldB;
    }
    store_sum4<NT>(sum + a_off, sa);
    store_sum4<NT>(sum + a_off + 256, sb);
    if (DEQ) {
        // the index words again (two registers live instead of eight indices)
        const auto k = [&](uint32_t word, int j) { return MULTI ? min((word >> (8 * j)) & 0xFFu, kmax) : 0u; };
        f32x4 oa, ob;
        oa.x = static_cast<float>(sa.x) * deq_t[k(in.ka, 0)];
        oa.y = static_cast<float>(sa.y) * deq_t[k(in.ka, 1)];
        oa.z = static_cast<float>(sa.z) * deq_t[k(in.ka, 2)];
        oa.w = static_cast<float>(sa.w) * deq_t[k(in.ka, 3)];
        ob.x = static_cast<float>(sb.x) * deq_t[k(in.kb, 0)];
        ob.y = static_cast<float>(sb.y) * deq_t[k(in.kb, 1)];
        ob.z = static_cast<float>(sb.z) * deq_t[k(in.kb, 2)];
        ob.w = static_cast<float>(sb.w) * deq_t[k(in.kb, 3)];
        store_nt(out + a_off, oa);
        store_nt(out + a_off + 256, ob);
    }
}

// The coordinates past the last whole tile (fewer than 512): lane t of one
// wave takes the 8 contiguous coordinates of group ntiles * 64 + t for every
// row, then stores their sums (and reconstruction).  inv_s holds s_k / W (not
// scaled).  NIB as for load_tile.
template <bool MULTI, bool ACC, bool DEQ, bool NIB = false>
__device__ __forceinline__ void quant_sum_tail(const float* __restrict__ g, int64_t d, int64_t ldg, int32_t rows,
                                               uint32_t worker0, const uint8_t* __restrict__ idx, int64_t ntiles,
                                               const float* inv_s, float inv0, float s0, uint32_t kmax,
                                               uint32_t key0, uint32_t key1, int32_t* __restrict__ sum,
                                               const float* deq_t, float* __restrict__ out)
{
    const int64_t q = (ntiles << 6) + (threadIdx.x & 63);
    const int64_t base = q << 3;
    if (base >= d)
        return;
    float inv[8];
    uint32_t kk[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const uint32_t raw = base + j < d ? (NIB ? nibble_at(idx, base + j) : static_cast<uint32_t>(idx[base + j])) : 0u;
        kk[j] = MULTI ? min(raw, kmax) : 0u;
        inv[j] = MULTI ? inv_s[kk[j]] : inv0;
    }
    int32_t acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    for (int32_t r = 0; r < rows; ++r) {
        const float* row = g + static_cast<int64_t>(r) * ldg;
        float v[8];
        int32_t code[8];
#pragma unroll
        for (int j = 0; j < 8; ++j)
            v[j] = base + j < d ? row[base + j] : 0.0f;
        quantise_group(v, inv, s0, static_cast<uint64_t>(q), worker0 + static_cast<uint32_t>(r), key0, key1, code);
#pragma unroll
        for (int j = 0; j < 8; ++j)
            acc[j] += code[j];
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        if (base + j < d) {
            const int32_t s = acc[j] + (ACC ? sum[base + j] : 0);
            sum[base + j] = s;
            if (DEQ)
                out[base + j] = static_cast<float>(s) * deq_t[kk[j]];
        }
    }
}

// ROW1: the one-row form (a streamed worker), compiled apart so that it does
// not carry the row loop's registers.  NIB: the index as 4-bit fields.
template <bool MULTI, bool ACC, bool DEQ, bool NT, bool ROW1, bool NIB>
__global__ __launch_bounds__(kBlock) void k_quant_sum(const float* __restrict__ g, int64_t d, int32_t rows,
                                                      int64_t ldg, int32_t worker0, const float* __restrict__ wptr,
                                                      ScaleSet S, const uint8_t* __restrict__ idx, uint32_t key0,
                                                      uint32_t key1, int32_t* __restrict__ sum, int32_t M,
                                                      float* __restrict__ out)
{
    __shared__ float inv_s[kMaxScales];  // s_k / W
    __shared__ float inv_p[kMaxScales];  // s_k / W * 2^16 when pre
    __shared__ float deq_s[kMaxScales];  // RN32(W / (M s_k))
    const int lane = threadIdx.x & 63;
    const int64_t ntiles = d >> 9;
    const int32_t wave_in_block = __builtin_amdgcn_readfirstlane(static_cast<int32_t>(threadIdx.x >> 6));
    const int64_t first = static_cast<int64_t>(blockIdx.x) * (kBlock / 64) + wave_in_block;
    const int64_t stride = static_cast<int64_t>(gridDim.x) * (kBlock / 64);
    const uint32_t w0 = static_cast<uint32_t>(worker0);

    // the first tile's loads (row 0, its index words, the old sums) go out
    // before W is read and the tables are formed
    TileIn in0 = {};
    i32x4 oldA0 = {0, 0, 0, 0}, oldB0 = {0, 0, 0, 0};
    if (first < ntiles) {
        const int64_t a_off = (first << 9) + 4 * lane;
        in0 = load_tile<MULTI, NIB>(g, idx, a_off);
        if (ACC) {
            oldA0 = load_sum4<NT>(sum + a_off);
            oldB0 = load_sum4<NT>(sum + a_off + 256);
        }
    }

    const float W = *wptr;
    const float q0 = div_rn32(S.s[0], W);
    const bool zero = zero_path(W, q0);
    const bool pre = zero || (MULTI ? div_rn32(S.s_last, W) : q0) <= 0x1p100f;
    if (threadIdx.x < S.K) {
        const float inv = zero ? 0.0f : div_rn32(S.s[threadIdx.x], W);
        inv_s[threadIdx.x] = inv;
        inv_p[threadIdx.x] = pre ? inv * 65536.0f : inv;
        if (DEQ) {
            const float denom = static_cast<float>(static_cast<double>(M) * static_cast<double>(S.s[threadIdx.x]));
            deq_s[threadIdx.x] = zero ? 0.0f : div_rn32(W, denom);
        }
    }
    __syncthreads();
    const float inv0 = zero ? 0.0f : q0;
    const float s0 = S.s[0];
    const uint32_t kmax = static_cast<uint32_t>(S.K - 1);
    uint32_t one2 = 0x00010001u;
    asm("" : "+s"(one2));

    // the preloaded tile, then (on a grid capped below one tile per wave)
    // every stride-th tile after it
    if (first < ntiles) {
        if (pre)
            quant_sum_tile<MULTI, true, ACC, DEQ, NT, ROW1>(g, ldg, rows, w0, first, in0, oldA0, oldB0, inv_p,
                                                      inv0 * 65536.0f, s0 * 65536.0f, kmax, key0, key1, one2, sum,
                                                      deq_s, out);
        else
            quant_sum_tile<MULTI, false, ACC, DEQ, NT, ROW1>(g, ldg, rows, w0, first, in0, oldA0, oldB0, inv_p, inv0, s0,
                                                       kmax, key0, key1, one2, sum, deq_s, out);
    }
    if (stride < ntiles) {
        for (int64_t T = first + stride; T < ntiles; T += stride) {
            const int64_t a_off = (T << 9) + 4 * lane;
            const TileIn in = load_tile<MULTI, NIB>(g, idx, a_off);
            i32x4 oldA = {0, 0, 0, 0}, oldB = {0, 0, 0, 0};
            if (ACC) {
                oldA = load_sum4<NT>(sum + a_off);
                oldB = load_sum4<NT>(sum + a_off + 256);
            }
            if (pre)
                quant_sum_tile<MULTI, true, ACC, DEQ, NT, ROW1>(g, ldg, rows, w0, T, in, oldA, oldB, inv_p, inv0 * 65536.0f,
                                                          s0 * 65536.0f, kmax, key0, key1, one2, sum, deq_s, out);
            else
                quant_sum_tile<MULTI, false, ACC, DEQ, NT, ROW1>(g, ldg, rows, w0, T, in, oldA, oldB, inv_p, inv0, s0,
                                                           kmax, key0, key1, one2, sum, deq_s, out);
        }
    }
    if (blockIdx.x == 0 && threadIdx.x < 64)
        quant_sum_tail<MULTI, ACC, DEQ, NIB>(g, d, ldg, rows, w0, idx, ntiles, inv_s, inv0, s0, kmax, key0, key1, sum,
                                        deq_s, out);
}

// ---------------------------------------------------------------------------
// The shared scale index formed inside the quantise-and-sum over all M <=
// kFuseRows rows (Sec. 3.2: Eq. (11) with scale sharing, then Eq. (12), the
// sum and Eq. (13)).  One wave per 512-coordinate tile, as k_quant_sum, but
// every row of the tile is loaded at once and held in registers: a
// coordinate's index comes from its exact largest usable |g| over the rows,
// and the rows are then quantised from registers, so neither the rows'
// maxima nor an index pass over them is needed.  The index uses the
// thresholds T_k of k_index_max (#{k : a <= T_k} - 1): when no binade holds
// two thresholds, a table over the exponent field gives, for binade e, the
// count above it and the bits of the one threshold inside it, and since the
// bits of non-negative binary32 values order like the values, a coordinate
// costs one lookup and one integer compare, exact with no ties to resolve.
// ROWS is M rounded up to a power of two; rows past M re-read row M - 1
// (no change to the maximum, no branch on the loads) and are not quantised.
// ---------------------------------------------------------------------------
// max(m, |x|, |y|) in one instruction (v_maximum3_f32, the absolute values
// by source modifiers).  This maximum propagates NaN: the result is NaN if
// any operand is, else infinite if any operand is, else the largest finite
// value, so a running maximum that stays finite saw finite values only.
__device__ __forceinline__ float max3_abs(float m, float x, float y)
{
    return __builtin_elementwise_maximum(m, __builtin_elementwise_maximum(fabsf(x), fabsf(y)));
}

// INDEX: form the tile's shared index (several scales) and store it; else
// one scale, every index 0.  The first `rows` rows are quantised, row r as
// worker worker0 + r.
// The shared index of a lane's eight coordinates of one tile (A quad, then B
// quad) from the largest usable |g| over the ROWS rows it holds: two rows per
// instruction with the NaN- and infinity-propagating maximum; a result that
// is not finite means some value was not usable (infinite or NaN), and then
// the lane forms the largest usable |g| value by value.  Then the exponent
// table (by_table) or K threshold compares.
template <int ROWS>
__device__ __forceinline__ void tile_index(const f32x4 (&A)[ROWS], const f32x4 (&B)[ROWS], const uint2* tab,
                                           bool by_table, const float* thr, int32_t K, bool zero, uint32_t k[8])
{
    float a[8] = {0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f};
    static_assert(ROWS % 2 == 0, "rows are taken in pairs");
#pragma unroll
    for (int r = 0; r < ROWS; r += 2) {
        a[0] = max3_abs(a[0], A[r].x, A[r + 1].x);
        a[1] = max3_abs(a[1], A[r].y, A[r + 1].y);
        a[2] = max3_abs(a[2], A[r].z, A[r + 1].z);
        a[3] = max3_abs(a[3], A[r].w, A[r + 1].w);
        a[4] = max3_abs(a[4], B[r].x, B[r + 1].x);
        a[5] = max3_abs(a[5], B[r].y, B[r + 1].y);
        a[6] = max3_abs(a[6], B[r].z, B[r + 1].z);
        a[7] = max3_abs(a[7], B[r].w, B[r + 1].w);
    }
    uint32_t worst = 0u;
#pragma unroll
    for (int j = 0; j < 8; ++j)
        worst = max(worst, __float_as_uint(a[j]));
    if (__builtin_expect(worst >= 0x7F800000u, 0)) {
#pragma unroll
        for (int j = 0; j < 8; ++j)
            a[j] = 0.0f;
#pragma unroll
        for (int r = 0; r < ROWS; ++r) {
            a[0] = fmaxf(a[0], usable_or_zero(A[r].x));
            a[1] = fmaxf(a[1], usable_or_zero(A[r].y));
            a[2] = fmaxf(a[2], usable_or_zero(A[r].z));
            a[3] = fmaxf(a[3], usable_or_zero(A[r].w));
            a[4] = fmaxf(a[4], usable_or_zero(B[r].x));
            a[5] = fmaxf(a[5], usable_or_zero(B[r].y));
            a[6] = fmaxf(a[6], usable_or_zero(B[r].z));
            a[7] = fmaxf(a[7], usable_or_zero(B[r].w));
        }
    }
    if (by_table) {
        const uint32_t kzero = static_cast<uint32_t>(K - 1);
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const uint32_t b = __float_as_uint(a[j]);
            const uint2 t = tab[b >> 23];
            k[j] = b != 0u ? t.x + (b <= t.y ? 1u : 0u) : kzero;
        }
    } else {
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            int32_t count = 0;
            for (int q = 0; q < K; ++q)
                count += a[j] <= thr[q] ? 1 : 0;
            k[j] = index_from_count(a[j], count, K, zero);
        }
    }
}

// Stores a lane's eight index bytes of one tile: the A quad's at a_off, the B
// quad's at a_off + 256.
template <bool NT>
__device__ __forceinline__ void store_index(uint8_t* __restrict__ idx, int64_t a_off, const uint32_t k[8])
{
    const uint32_t ka = k[0] | (k[1] << 8) | (k[2] << 16) | (k[3] << 24);
    const uint32_t kb = k[4] | (k[5] << 8) | (k[6] << 16) | (k[7] << 24);
    uint32_t* ip = reinterpret_cast<uint32_t*>(idx + a_off);
    if (NT) {
        __builtin_nontemporal_store(ka, ip);
        __builtin_nontemporal_store(kb, ip + 64);
    } else {
        ip[0] = ka;
        ip[64] = kb;
    }
}

template <int ROWS, bool PRE, bool NT, bool INDEX>
__device__ __forceinline__ void index_quant_sum_tile(const f32x4 (&A)[ROWS], const f32x4 (&B)[ROWS], int32_t rows,
                                                     uint32_t worker0, int64_t T, const uint2* tab, bool by_table,
                                                     const float* thr, int32_t K, bool zero, const float* inv_t,
                                                     float s0x, const float* deq_t, uint32_t key0, uint32_t key1,
                                                     uint32_t one2, uint8_t* __restrict__ idx,
                                                     int32_t* __restrict__ sum, float* __restrict__ out)
{
    const int lane = threadIdx.x & 63;
    const int64_t a_off = (T << 9) + 4 * lane;
    uint32_t k[8] = {0u, 0u, 0u, 0u, 0u, 0u, 0u, 0u};
    if (INDEX) {
        tile_index<ROWS>(A, B, tab, by_table, thr, K, zero, k);
        store_index<NT>(idx, a_off, k);
    }
    float inv[8];
#pragma unroll
    for (int j = 0; j < 8; ++j)
        inv[j] = inv_t[k[j]];
    uint32_t h[4] = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int r = 0; r < ROWS; ++r) {
        if (r < rows) {
            const float v[8] = {A[r].x, A[r].y, A[r].z, A[r].w, B[r].x, B[r].y, B[r].z, B[r].w};
            uint32_t p[4];
            tile_codes<PRE>(v, inv, s0x, T, worker0 + static_cast<uint32_t>(r), key0, key1, one2, p);
#pragma unroll
            for (int j = 0; j < 4; ++j)
                h[j] = __builtin_bit_cast(uint32_t, __builtin_bit_cast(u16x2, h[j]) + __builtin_bit_cast(u16x2, p[j]));
        }
    }
    int32_t acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    widen_pairs(h, acc);
    const i32x4 sa = {acc[0], acc[1], acc[2], acc[3]};
    const i32x4 sb = {acc[4], acc[5], acc[6], acc[7]};
    store_sum4<NT>(sum + a_off, sa);
    store_sum4<NT>(sum + a_off + 256, sb);
    f32x4 oa, ob;
    oa.x = static_cast<float>(sa.x) * deq_t[k[0]];
    oa.y = static_cast<float>(sa.y) * deq_t[k[1]];
    oa.z = static_cast<float>(sa.z) * deq_t[k[2]];
    oa.w = static_cast<float>(sa.w) * deq_t[k[3]];
    ob.x = static_cast<float>(sb.x) * deq_t[k[4]];
    ob.y = static_cast<float>(sb.y) * deq_t[k[5]];
    ob.z = static_cast<float>(sb.z) * deq_t[k[6]];
    ob.w = static_cast<float>(sb.w) * deq_t[k[7]];
    store_nt(out + a_off, oa);
    store_nt(out + a_off + 256, ob);
}

// The coordinates past the last whole tile (fewer than 512): lane t of one
// wave takes the 8 contiguous coordinates of group ntiles * 64 + t, forms
// their indices from the rows' maxima (threshold counts), then quantises and
// sums every row.  inv_s holds s_k / W (not scaled).
__device__ __forceinline__ void index_quant_sum_tail(const float* __restrict__ g, int64_t d, int64_t ldg, int32_t M,
                                                     int64_t ntiles, const float* thr, int32_t K, bool zero,
                                                     const float* inv_s, float s0, uint32_t key0, uint32_t key1,
                                                     uint8_t* __restrict__ idx, int32_t* __restrict__ sum,
                                                     const float* deq_t, float* __restrict__ out)
{
    const int64_t q = (ntiles << 6) + (threadIdx.x & 63);
    const int64_t base = q << 3;
    if (base >= d)
        return;
    float a[8] = {0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f};
    for (int32_t r = 0; r < M; ++r) {
        const float* row = g + static_cast<int64_t>(r) * ldg;
#pragma unroll
        for (int j = 0; j < 8; ++j)
            a[j] = fmaxf(a[j], usable_or_zero(base + j < d ? row[base + j] : 0.0f));
    }
    uint32_t kk[8];
    float inv[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        int32_t count = 0;
        for (int k = 0; k < K; ++k)
            count += a[j] <= thr[k] ? 1 : 0;
        kk[j] = index_from_count(a[j], count, K, zero);
        inv[j] = inv_s[kk[j]];
    }
    int32_t acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    for (int32_t r = 0; r < M; ++r) {
        const float* row = g + static_cast<int64_t>(r) * ldg;
        float v[8];
        int32_t code[8];
#pragma unroll
        for (int j = 0; j < 8; ++j)
            v[j] = base + j < d ? row[base + j] : 0.0f;
        quantise_group(v, inv, s0, static_cast<uint64_t>(q), static_cast<uint32_t>(r), key0, key1, code);
#pragma unroll
        for (int j = 0; j < 8; ++j)
            acc[j] += code[j];
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        if (base + j < d) {
            idx[base + j] = static_cast<uint8_t>(kk[j]);
            sum[base + j] = acc[j];
            out[base + j] = static_cast<float>(acc[j]) * deq_t[kk[j]];
        }
    }
}

template <int ROWS, bool NT>
__global__ __launch_bounds__(kBlock) void k_index_quant_sum(const float* __restrict__ g, int64_t d, int32_t M,
                                                            int64_t ldg, const float* __restrict__ wptr, ScaleSet S,
                                                            uint32_t key0, uint32_t key1, uint8_t* __restrict__ idx,
                                                            int32_t* __restrict__ sum, float* __restrict__ out)
{
    __shared__ float inv_s[kMaxScales];  // s_k / W
    __shared__ float inv_p[kMaxScales];  // s_k / W * 2^16 when pre
    __shared__ float deq_s[kMaxScales];  // RN32(W / (M s_k))
    __shared__ float thr_s[kMaxScales];  // T_k
    __shared__ uint2 tab_s[256];
    const int lane = threadIdx.x & 63;
    const int64_t ntiles = d >> 9;
    const int32_t wave_in_block = __builtin_amdgcn_readfirstlane(static_cast<int32_t>(threadIdx.x >> 6));
    const int64_t first = static_cast<int64_t>(blockIdx.x) * (kBlock / 64) + wave_in_block;
    const int64_t stride = static_cast<int64_t>(gridDim.x) * (kBlock / 64);

    // every row of the first tile goes out before W is read and the tables
    // are formed
    f32x4 A[ROWS], B[ROWS];
    const auto load_rows = [&](int64_t T) {
        const int64_t a_off = (T << 9) + 4 * lane;
#pragma unroll
        for (int r = 0; r < ROWS; ++r) {
            const float* row = g + static_cast<int64_t>(r < M ? r : M - 1) * ldg;
            A[r] = load_nt(row + a_off);
            B[r] = load_nt(row + a_off + 256);
        }
    };
    if (first < ntiles)
        load_rows(first);

    const float W = *wptr;
    const float s0 = S.s[0];
    const int32_t K = S.K;
    const float q0 = div_rn32(s0, W);
    const bool zero = zero_path(W, q0);
    const bool pre = zero || div_rn32(S.s_last, W) <= 0x1p100f;
    if (threadIdx.x < K) {
        const float inv = zero ? 0.0f : div_rn32(S.s[threadIdx.x], W);
        inv_s[threadIdx.x] = inv;
        inv_p[threadIdx.x] = pre ? inv * 65536.0f : inv;
        const float denom = static_cast<float>(static_cast<double>(M) * static_cast<double>(S.s[threadIdx.x]));
        deq_s[threadIdx.x] = zero ? 0.0f : div_rn32(W, denom);
        thr_s[threadIdx.x] = zero ? 0.0f : index_threshold(inv, s0);
    }
    __syncthreads();
    // thread e forms the table's entry e (the rule of k_index_max with the
    // thresholds' full bits): x + [bits(a) <= y] is the index of a value a > 0
    // of binade e; a binade without a threshold inside holds y = 0xFFFFFFFF
    // with x lowered by one; on the zero path every value gets K - 1
    int crowded = 0;
    {
        const uint32_t e = threadIdx.x;
        int32_t above = 0, inside = 0;
        uint32_t tin = 0u;
        for (int k = 0; k < K; ++k) {
            const uint32_t tb = __float_as_uint(thr_s[k]);
            above += (tb >> 23) > e ? 1 : 0;
            if ((tb >> 23) == e) {
                ++inside;
                tin = tb;
            }
        }
        uint2 ent;
        if (zero) {
            ent.x = static_cast<uint32_t>(K - 2);
            ent.y = 0xFFFFFFFFu;
        } else {
            crowded = inside > 1 ? 1 : 0;
            const bool limit = inside > 0 && above > 0;
            ent.x = static_cast<uint32_t>(above > 0 ? above - 1 : 0) - (limit ? 0u : 1u);
            ent.y = limit ? tin : 0xFFFFFFFFu;
        }
        tab_s[e] = ent;
    }
    const bool by_table = __syncthreads_or(crowded) == 0;
    uint32_t one2 = 0x00010001u;
    asm("" : "+s"(one2));
    const float s0x = pre ? s0 * 65536.0f : s0;

    // the preloaded tile, then (on a grid capped below one tile per wave)
    // every stride-th tile after it
    for (int64_t T = first; T < ntiles; T += stride) {
        if (T != first)
            load_rows(T);
        if (pre)
            index_quant_sum_tile<ROWS, true, NT, true>(A, B, M, 0u, T, tab_s, by_table, thr_s, K, zero, inv_p, s0x,
                                                       deq_s, key0, key1, one2, idx, sum, out);
        else
            index_quant_sum_tile<ROWS, false, NT, true>(A, B, M, 0u, T, tab_s, by_table, thr_s, K, zero, inv_p, s0x,
                                                        deq_s, key0, key1, one2, idx, sum, out);
    }
    if (blockIdx.x == 0 && threadIdx.x < 64)
        index_quant_sum_tail(g, d, ldg, M, ntiles, thr_s, K, zero, inv_s, s0, key0, key1, idx, sum, deq_s, out);
}

// ---------------------------------------------------------------------------
// The shared index formed in the quantiser (several scales, at most 16 rows,
// codes stored): k_index_quant_sum's tiles, every row of a tile held by one
// wave and the index formed from their exact maxima and stored, with each
// row's codes stored (int8, or packed 4- or 2-bit fields) instead of summed.
// The codes and the index equal uq_shared_scale's index followed by the
// quantiser's codes, given the same W.  A wave collects its rows' codes of
// the tile in LDS and stores them as 16-byte pieces: at VGG-16 size with
// 4-bit codes 1.85 ms against 1.96 for two 2-byte stores per lane and row.
// ---------------------------------------------------------------------------
// Four consecutive codes (16-bit lanes of p01, p23) in the code row's layout:
// 4, 2 or 1 bytes.
template <int BITS>
__device__ __forceinline__ uint32_t pack_quad(uint32_t p01, uint32_t p23)
{
    const uint32_t w = __builtin_amdgcn_perm(p23, p01, 0x06040200u);
    if (BITS == 8)
        return w;
    if (BITS == 4) {
        const uint32_t x = w & 0x0F0F0F0Fu;
        const uint32_t y = x | (x >> 4);
        return __builtin_amdgcn_perm(0u, y, 0x0C0C0200u);
    }
    const uint32_t x = w & 0x03030303u;
    const uint32_t y = x | (x >> 6);
    return (y | (y >> 12)) & 0xFFu;
}

template <int BITS>
__device__ __forceinline__ void lds_put(uint8_t* p, uint32_t v)
{
    if (BITS == 8)
        *reinterpret_cast<uint32_t*>(p) = v;
    else if (BITS == 4)
        *reinterpret_cast<uint16_t*>(p) = static_cast<uint16_t>(v);
    else
        *p = static_cast<uint8_t>(v);
}

template <int ROWS, int BITS, bool PRE, bool NT>
__device__ __forceinline__ void index_quantise_tile(const f32x4 (&A)[ROWS], const f32x4 (&B)[ROWS], int32_t rows,
                                                    int64_t T, const uint2* tab, bool by_table, const float* thr,
                                                    int32_t K, bool zero, const float* inv_t, float s0x,
                                                    uint32_t key0, uint32_t key1, uint32_t one2,
                                                    uint8_t* __restrict__ idx, uint8_t* __restrict__ codes,
                                                    int64_t ldc, uint8_t* stage)
{
    const int lane = threadIdx.x & 63;
    const int64_t a_off = (T << 9) + 4 * lane;
    uint32_t k[8];
    tile_index<ROWS>(A, B, tab, by_table, thr, K, zero, k);
    store_index<NT>(idx, a_off, k);
    float inv[8];
#pragma unroll
    for (int j = 0; j < 8; ++j)
        inv[j] = inv_t[k[j]];
#pragma unroll
    for (int r = 0; r < ROWS; ++r) {
        if (r < rows) {
            const float v[8] = {A[r].x, A[r].y, A[r].z, A[r].w, B[r].x, B[r].y, B[r].z, B[r].w};
            uint32_t p[4];
            tile_codes<PRE>(v, inv, s0x, T, static_cast<uint32_t>(r), key0, key1, one2, p);
            // the row's codes of this tile into the wave's LDS rows
            uint8_t* srow = stage + r * (64 * BITS);
            lds_put<BITS>(srow + (4 * lane) * BITS / 8, pack_quad<BITS>(p[0], p[1]));
            lds_put<BITS>(srow + (256 + 4 * lane) * BITS / 8, pack_quad<BITS>(p[2], p[3]));
        }
    }
    // 16-byte pieces of the wave's rows (64 * BITS bytes per row and tile),
    // several rows' pieces per store: the wave's own LDS writes above
    // complete before these reads
    constexpr int kPieces = 64 * BITS / 16;
    constexpr int kAll = ROWS * kPieces;
    __asm__ volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
    for (int c0 = 0; c0 < kAll; c0 += 64) {
        const int c = c0 + lane;
        const int r = c / kPieces;
        const int off = (c % kPieces) * 16;
        if (c < kAll && r < rows) {
            const u32x4 v = *reinterpret_cast<const u32x4*>(stage + r * (64 * BITS) + off);
            u32x4* dst = reinterpret_cast<u32x4*>(codes + static_cast<int64_t>(r) * ldc + T * (64 * BITS) + off);
            if (NT)
                __builtin_nontemporal_store(v, dst);
            else
                *dst = v;
        }
    }
}

// The coordinates past the last whole tile (fewer than 512): lane t of one
// wave takes the 8 contiguous coordinates of group ntiles * 64 + t, forms
// their indices from the rows' maxima (threshold counts), then quantises and
// stores every row's codes.  inv_s holds s_k / W (not scaled).
template <int BITS>
__device__ __forceinline__ void index_quantise_tail(const float* __restrict__ g, int64_t d, int64_t ldg, int32_t M,
                                                    int64_t ntiles, const float* thr, int32_t K, bool zero,
                                                    const float* inv_s, float s0, uint32_t key0, uint32_t key1,
                                                    uint8_t* __restrict__ idx, uint8_t* __restrict__ codes,
                                                    int64_t ldc)
{
    const int64_t q = (ntiles << 6) + (threadIdx.x & 63);
    const int64_t base = q << 3;
    if (base >= d)
        return;
    float a[8] = {0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f};
    for (int32_t r = 0; r < M; ++r) {
        const float* row = g + static_cast<int64_t>(r) * ldg;
#pragma unroll
        for (int j = 0; j < 8; ++j)
            a[j] = fmaxf(a[j], usable_or_zero(base + j < d ? row[base + j] : 0.0f));
    }
    float inv[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        int32_t count = 0;
        for (int k = 0; k < K; ++k)
            count += a[j] <= thr[k] ? 1 : 0;
        const uint32_t kk = index_from_count(a[j], count, K, zero);
        inv[j] = inv_s[kk];
        if (base + j < d)
            idx[base + j] = static_cast<uint8_t>(kk);
    }
    for (int32_t r = 0; r < M; ++r) {
        const float* row = g + static_cast<int64_t>(r) * ldg;
        uint8_t* out = codes + static_cast<int64_t>(r) * ldc;
        float v[8];
        int32_t code[8];
#pragma unroll
        for (int j = 0; j < 8; ++j)
            v[j] = base + j < d ? row[base + j] : 0.0f;
        quantise_group(v, inv, s0, static_cast<uint64_t>(q), static_cast<uint32_t>(r), key0, key1, code);
        if (BITS == 8) {
#pragma unroll
            for (int j = 0; j < 8; ++j)
                if (base + j < d)
                    out[base + j] = static_cast<uint8_t>(code[j]);
        } else if (BITS == 4) {
            // the group's 8 codes fill whole bytes of its own (codes past d are 0)
            *reinterpret_cast<uint32_t*>(out + base / 2) = pack_field<4>(code) | (pack_field<4>(code + 4) << 16);
        } else {
            *reinterpret_cast<uint16_t*>(out + base / 4) =
                static_cast<uint16_t>(pack_field<2>(code) | (pack_field<2>(code + 4) << 8));
        }
    }
}

template <int ROWS, int BITS, bool NT>
__global__ __launch_bounds__(kBlock) void k_index_quantise(const float* __restrict__ g, int64_t d, int32_t M,
                                                           int64_t ldg, const float* __restrict__ wptr, ScaleSet S,
                                                           uint32_t key0, uint32_t key1, uint8_t* __restrict__ idx,
                                                           uint8_t* __restrict__ codes, int64_t ldc)
{
    __shared__ float inv_s[kMaxScales];  // s_k / W
    __shared__ float inv_p[kMaxScales];  // s_k / W * 2^16 when pre
    __shared__ float thr_s[kMaxScales];  // T_k
    __shared__ uint2 tab_s[256];
    __shared__ __align__(16) uint8_t stage_s[4][ROWS * 64 * BITS];  // each wave's code rows of its tile
    const int lane = threadIdx.x & 63;
    const int64_t ntiles = d >> 9;
    const int32_t wave_in_block = __builtin_amdgcn_readfirstlane(static_cast<int32_t>(threadIdx.x >> 6));
    const int64_t first = static_cast<int64_t>(blockIdx.x) * (kBlock / 64) + wave_in_block;
    const int64_t stride = static_cast<int64_t>(gridDim.x) * (kBlock / 64);
    uint8_t* stage = stage_s[wave_in_block];

    // every row of the first tile goes out before W is read and the tables
    // are formed
    f32x4 A[ROWS], B[ROWS];
    const auto load_rows = [&](int64_t T) {
        const int64_t a_off = (T << 9) + 4 * lane;
#pragma unroll
        for (int r = 0; r < ROWS; ++r) {
            const float* row = g + static_cast<int64_t>(r < M ? r : M - 1) * ldg;
            A[r] = load_nt(row + a_off);
            B[r] = load_nt(row + a_off + 256);
        }
    };
    if (first < ntiles)
        load_rows(first);

    const float W = *wptr;
    const float s0 = S.s[0];
    const int32_t K = S.K;
    const float q0 = div_rn32(s0, W);
    const bool zero = zero_path(W, q0);
    const bool pre = zero || div_rn32(S.s_last, W) <= 0x1p100f;
    if (threadIdx.x < K) {
        const float inv = zero ? 0.0f : div_rn32(S.s[threadIdx.x], W);
        inv_s[threadIdx.x] = inv;
        inv_p[threadIdx.x] = pre ? inv * 65536.0f : inv;
        thr_s[threadIdx.x] = zero ? 0.0f : index_threshold(inv, s0);
    }
    __syncthreads();
    // thread e forms the table's entry e, as in k_index_quant_sum
    int crowded = 0;
    {
        const uint32_t e = threadIdx.x;
        int32_t above = 0, inside = 0;
        uint32_t tin = 0u;
        for (int k = 0; k < K; ++k) {
            const uint32_t tb = __float_as_uint(thr_s[k]);
            above += (tb >> 23) > e ? 1 : 0;
            if ((tb >> 23) == e) {
                ++inside;
                tin = tb;
            }
        }
        uint2 ent;
        if (zero) {
            ent.x = static_cast<uint32_t>(K - 2);
            ent.y = 0xFFFFFFFFu;
        } else {
            crowded = inside > 1 ? 1 : 0;
            const bool limit = inside > 0 && above > 0;
            ent.x = static_cast<uint32_t>(above > 0 ? above - 1 : 0) - (limit ? 0u : 1u);
            ent.y = limit ? tin : 0xFFFFFFFFu;
        }
        tab_s[e] = ent;
    }
    const bool by_table = __syncthreads_or(crowded) == 0;
    uint32_t one2 = 0x00010001u;
    asm("" : "+s"(one2));
    const float s0x = pre ? s0 * 65536.0f : s0;

    for (int64_t T = first; T < ntiles; T += stride) {
        if (T != first)
            load_rows(T);
        if (pre)
            index_quantise_tile<ROWS, BITS, true, NT>(A, B, M, T, tab_s, by_table, thr_s, K, zero, inv_p, s0x,
                                                             key0, key1, one2, idx, codes, ldc, stage);
        else
            index_quantise_tile<ROWS, BITS, false, NT>(A, B, M, T, tab_s, by_table, thr_s, K, zero, inv_p, s0x,
                                                              key0, key1, one2, idx, codes, ldc, stage);
    }
    if (blockIdx.x == 0 && threadIdx.x < 64)
        index_quantise_tail<BITS>(g, d, ldg, M, ntiles, thr_s, K, zero, inv_s, s0, key0, key1, idx, codes, ldc);
}

// ---------------------------------------------------------------------------
// One scale, 5 to 16 rows set and reconstructed in one call, the rows of a
// tile split over the block's four waves: wave w holds rows w, w + 4, ...
// (RPW of them) of the block's 512-coordinate tile in k_quantise's lane
// layout, codes them (the codes and draws of k_quantise for that row and
// tile) and sums them in the 16-bit lanes of the pair registers; the waves'
// int32 sums meet in LDS, and waves 0 and 1 add them and store the tile's A
// and B quads of sums and of the reconstruction.  The integer sums are exact
// in any order.  Against one wave holding every row of a tile (the layout
// k_index_quant_sum keeps for several scales), a wave needs about a third of
// the registers (86 against 217 for 16 rows), so five waves share a SIMD
// instead of two and hide each other's loads: measured on MI355X, 1.76 ->
// 1.62 ms at VGG-16 size (16 rows) and 72.9 -> 69.6 us at ResNet-18 size
// (8 rows, against k_quant_sum's row loop).  The same split with the shared
// index formed in the pass (the waves' maxima meeting in LDS first) was
// slower with several scales: each tile then waits at two barriers and each
// block forms the thresholds and the exponent table again (ResNet-50 size,
// 8 rows: 0.237 against 0.175 ms; VGG-16, four scales: 1.94 against 1.79 ms;
// 0.209 and 1.82 ms with four tiles per block).
// ---------------------------------------------------------------------------
template <int RPW, bool PRE, bool NT>
__device__ __forceinline__ void split_tile(const f32x4 (&A)[RPW], const f32x4 (&B)[RPW], int32_t rows,
                                           uint32_t worker0, int64_t T, float inv0, float s0x, float deq0,
                                           uint32_t key0, uint32_t key1, uint32_t one2, i32x4 (*ps)[128],
                                           int32_t* __restrict__ sum, float* __restrict__ out)
{
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(static_cast<int32_t>(threadIdx.x >> 6));
    const int64_t a_off = (T << 9) + 4 * lane;
    const float inv[8] = {inv0, inv0, inv0, inv0, inv0, inv0, inv0, inv0};
    uint32_t h[4] = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int r = 0; r < RPW; ++r) {
        const int32_t m = wave + 4 * r;
        if (m < rows) {
            const float v[8] = {A[r].x, A[r].y, A[r].z, A[r].w, B[r].x, B[r].y, B[r].z, B[r].w};
            uint32_t p[4];
            tile_codes<PRE>(v, inv, s0x, T, worker0 + static_cast<uint32_t>(m), key0, key1, one2, p);
#pragma unroll
            for (int j = 0; j < 4; ++j)
                h[j] = __builtin_bit_cast(uint32_t, __builtin_bit_cast(u16x2, h[j]) + __builtin_bit_cast(u16x2, p[j]));
        }
    }
    int32_t acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    widen_pairs(h, acc);
    ps[wave][lane] = i32x4{acc[0], acc[1], acc[2], acc[3]};
    ps[wave][64 + lane] = i32x4{acc[4], acc[5], acc[6], acc[7]};
    __syncthreads();
    if (wave < 2) {
        // wave 0: the A quad of every lane, wave 1: the B quad
        const int q = 64 * wave + lane;
        const i32x4 s = (ps[0][q] + ps[1][q]) + (ps[2][q] + ps[3][q]);
        const int64_t off = a_off + 256 * wave;
        store_sum4<NT>(sum + off, s);
        f32x4 o;
        o.x = static_cast<float>(s.x) * deq0;
        o.y = static_cast<float>(s.y) * deq0;
        o.z = static_cast<float>(s.z) * deq0;
        o.w = static_cast<float>(s.w) * deq0;
        store_nt(out + off, o);
    }
}

// One block per tile (blocks stride over the tiles on a capped grid).
template <int RPW, bool NT>
__global__ __launch_bounds__(kBlock) void k_quant_sum_split(const float* __restrict__ g, int64_t d, int32_t rows,
                                                            int64_t ldg, int32_t worker0,
                                                            const float* __restrict__ wptr, ScaleSet S, uint32_t key0,
                                                            uint32_t key1, int32_t* __restrict__ sum, int32_t M,
                                                            float* __restrict__ out)
{
    __shared__ i32x4 ps_s[2][4][128];  // by tile parity: the next tile's sums never overwrite ones being read
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(static_cast<int32_t>(threadIdx.x >> 6));
    const int64_t ntiles = d >> 9;
    const uint32_t w0 = static_cast<uint32_t>(worker0);
    const int64_t first = blockIdx.x;

    // the first tile's rows go out before W is read
    f32x4 A[RPW], B[RPW];
    const auto load_rows = [&](int64_t T) {
        const int64_t a_off = (T << 9) + 4 * lane;
#pragma unroll
        for (int r = 0; r < RPW; ++r) {
            const int32_t m = wave + 4 * r;
            const float* row = g + static_cast<int64_t>(m < rows ? m : rows - 1) * ldg;
            A[r] = load_nt(row + a_off);
            B[r] = load_nt(row + a_off + 256);
        }
    };
    if (first < ntiles)
        load_rows(first);

    const float W = *wptr;
    const float s0 = S.s[0];
    const float q0 = div_rn32(s0, W);
    const bool zero = zero_path(W, q0);
    const bool pre = zero || q0 <= 0x1p100f;
    const float inv0 = zero ? 0.0f : q0;
    const float denom = static_cast<float>(static_cast<double>(M) * static_cast<double>(s0));
    const float deq0 = zero ? 0.0f : div_rn32(W, denom);
    uint32_t one2 = 0x00010001u;
    asm("" : "+s"(one2));
    const float s0x = pre ? s0 * 65536.0f : s0;
    const float invx = pre ? inv0 * 65536.0f : inv0;

    int parity = 0;
    for (int64_t T = first; T < ntiles; T += gridDim.x) {
        if (T != first)
            load_rows(T);
        if (pre)
            split_tile<RPW, true, NT>(A, B, rows, w0, T, invx, s0x, deq0, key0, key1, one2, ps_s[parity], sum, out);
        else
            split_tile<RPW, false, NT>(A, B, rows, w0, T, invx, s0x, deq0, key0, key1, one2, ps_s[parity], sum, out);
        parity ^= 1;
    }
    if (blockIdx.x == 0 && threadIdx.x < 64) {
        const float inv_t[1] = {inv0}, deq_t[1] = {deq0};
        quant_sum_tail<false, false, true>(g, d, ldg, rows, w0, nullptr, ntiles, inv_t, inv0, s0, 0u, key0, key1, sum,
                                           deq_t, out);
    }
}

// ---------------------------------------------------------------------------
// Host-side launchers (called by the ABI layer after validation).
// ---------------------------------------------------------------------------
// Tiles per wave for the quantiser.  Launch-shape sweeps on MI355X with cold
// caches: one tile per wave (a one-shot grid) is fastest for one scale; with
// several scales two consecutive tiles per wave amortise the per-block table
// set-up and read the shared index in longer runs.
// The quantiser stores its codes nontemporally when one launch writes more
// than this many bytes: measured 3% faster steps at VGG-16 size (2.2 GB of
// codes), 1.8-2.5% slower at ResNet-18 and ResNet-50 sizes (89 and 204 MB),
// where the sum then finds the codes in the 256 MB Infinity Cache.
constexpr int64_t kCodesNontemporalBytes = int64_t(512) << 20;

static int32_t quantise_tiles_per_wave(int32_t K)
{
    return K > 1 ? 2 : 1;
}

// Enough blocks for every unit to get its own thread / wave / tile (the
// streaming kernels run fastest as one pass with no grid-stride reuse).  The
// dispatch packet counts work-items in 32 bits, so the grid is capped at 2^22
// blocks; every kernel strides over whatever the grid does not cover.  Tests
// lower the cap to reach those strides at small sizes.
constexpr int64_t kMaxBlocks = int64_t(1) << 22;
static std::atomic<int64_t> g_one_shot_cap{kMaxBlocks};

bool set_one_shot_cap(int64_t blocks)
{
    if (blocks == 0)
        blocks = kMaxBlocks;
    if (blocks < kMinOneShotCap || blocks > kMaxBlocks)
        return false;
    g_one_shot_cap.store(blocks, std::memory_order_relaxed);
    return true;
}

static int64_t one_shot_cap()
{
    return g_one_shot_cap.load(std::memory_order_relaxed);
}

static unsigned one_shot(int64_t units, int64_t per_block)
{
    const int64_t cap = one_shot_cap();
    int64_t blocks = (units + per_block - 1) / per_block;
    blocks = blocks < 1 ? 1 : (blocks > cap ? cap : blocks);
    return static_cast<unsigned>(blocks);
}

// The fused pass stores the row maxima's keys nontemporally when they exceed
// this many bytes: measured 5% faster (the shared scale) at VGG-16 size
// (277 MB of keys), 3% slower at ResNet-50 size (51 MB), where the index pass
// reads them back from the 256 MB Infinity Cache.
constexpr int64_t kMaximaNontemporalBytes = int64_t(128) << 20;
// The index pass stores the index (one byte per coordinate) nontemporally
// beyond this many bytes, where the passes that read it back find it in HBM.
constexpr int64_t kIndexNontemporalBytes = int64_t(256) << 20;

hipError_t launch_shared_scale(const float* g, int64_t d, int32_t M, int64_t ldg, const ScaleSet& S,
                               float* w, uint8_t* idx, void* ws, hipStream_t stream, int32_t idx_bits)
{
    const bool nib = idx_bits == 4;
    if (use_fused(d, M, S.K)) {
        const FusedPlan plan = fused_plan(d);
        const FusedLayout L = fused_layout(d, M);
        double* part = static_cast<double*>(ws);
        double* sub = reinterpret_cast<double*>(static_cast<char*>(ws) + L.sub_off);
        double* rows = reinterpret_cast<double*>(static_cast<char*>(ws) + L.rows_off);
        IndexTables* tabs = reinterpret_cast<IndexTables*>(static_cast<char*>(ws) + L.tab_off);
        uint16_t* keys = fused_keys(ws, L);
        const dim3 grid(one_shot(plan.ntiles + 1, 1));
        // keys beyond half the 256 MB Infinity Cache are stored
        // nontemporally (the index pass would not find them there)
        const bool nt = 2 * d > kMaximaNontemporalBytes;
        const bool one = static_cast<int64_t>(grid.x) >= plan.ntiles + 1;
#define UQ_LAUNCH_NORM_MAX_(R, NT)                                                                                \
    do {                                                                                                          \
        if (one)                                                                                                  \
            hipLaunchKernelGGL((k_norm_max<R, NT, true>), grid, dim3(kBlock), 0, stream, g, d, M, ldg,            \
                               plan.ntiles, part, keys);                                                          \
        else                                                                                                      \
            hipLaunchKernelGGL((k_norm_max<R, NT, false>), grid, dim3(kBlock), 0, stream, g, d, M, ldg,           \
                               plan.ntiles, part, keys);                                                          \
    } while (0)
#define UQ_LAUNCH_NORM_MAX(R)              \
    do {                                   \
        if (nt)                            \
            UQ_LAUNCH_NORM_MAX_(R, true);  \
        else                               \
            UQ_LAUNCH_NORM_MAX_(R, false); \
    } while (0)
        if (M <= 4)
            UQ_LAUNCH_NORM_MAX(4);
        else if (M <= 8)
            UQ_LAUNCH_NORM_MAX(8);
        else
            UQ_LAUNCH_NORM_MAX(kFuseRows);
#undef UQ_LAUNCH_NORM_MAX
#undef UQ_LAUNCH_NORM_MAX_
        // the rows' sums: kRowsumSpan tile partials at a time, then those sums
        hipLaunchKernelGGL(k_rowsum, dim3(static_cast<unsigned>(plan.nsub), static_cast<unsigned>(M)), dim3(kBlock),
                           0, stream, part, plan.ntiles + 1, kRowsumSpan, sub);
        // then S_m, W and the index pass's constants in one block
        hipLaunchKernelGGL(k_index_prep, dim3(1), dim3(kBlock), 0, stream, sub, plan.nsub, M, rows, w, S, tabs);
        const unsigned gx = one_shot((d + 7) / 8, kIndexTile);
#define UQ_LAUNCH_INDEX_MAX(NT, NIB)                                                                            \
    hipLaunchKernelGGL((k_index_max<NT, NIB>), dim3(gx), dim3(kBlock), 0, stream, keys, g, ldg, d, M, tabs, S.K, idx)
        // the index is stored nontemporally beyond kIndexNontemporalBytes
        if ((nib ? (d + 1) / 2 : d) > kIndexNontemporalBytes) {
            if (nib) UQ_LAUNCH_INDEX_MAX(true, true); else UQ_LAUNCH_INDEX_MAX(true, false);
        } else {
            if (nib) UQ_LAUNCH_INDEX_MAX(false, true); else UQ_LAUNCH_INDEX_MAX(false, false);
        }
#undef UQ_LAUNCH_INDEX_MAX
        return hipGetLastError();
    }
    double* part = static_cast<double*>(ws);
    const NormPlan plan = norm_plan(d);
    if (plan.nchunks > 0) {
        // rows beyond the grid cap / nchunks are taken in turn by the same blocks
        int64_t gy = one_shot_cap() / plan.nchunks;
        gy = gy < 1 ? 1 : (gy > M ? M : gy);
        dim3 grid(static_cast<unsigned>(plan.nchunks), static_cast<unsigned>(gy));
        hipLaunchKernelGGL(k_sumsq, grid, dim3(kBlock), 0, stream, g, d, M, ldg, plan.chunk, plan.nchunks, part);
    }
    hipLaunchKernelGGL(k_finish, dim3(1), dim3(kFinishThreads), 0, stream, part, plan.nchunks, M, w);
    if (S.K > 1 && d > 0) {
        const unsigned gx = one_shot((d + 3) / 4, kBlock);
        if (nib)
            hipLaunchKernelGGL(k_index<true>, dim3(gx), dim3(kBlock), 0, stream, g, d, M, ldg, w, S, idx);
        else
            hipLaunchKernelGGL(k_index<false>, dim3(gx), dim3(kBlock), 0, stream, g, d, M, ldg, w, S, idx);
    }
    return hipGetLastError();
}

hipError_t launch_quantise(const float* g, int64_t d, int32_t rows, int64_t ldg, int32_t worker0,
                           const float* w, const ScaleSet& S, const uint8_t* idx, uint64_t seed,
                           void* codes, int64_t ldc, int32_t bits, hipStream_t stream)
{
    if (d == 0)
        return hipSuccess;
    const uint32_t key0 = static_cast<uint32_t>(seed);
    const uint32_t key1 = static_cast<uint32_t>(seed >> 32);
    // `tpw` consecutive 512-coordinate tiles per wave, four waves per block
    const int32_t tpw = quantise_tiles_per_wave(S.K);
    unsigned tile_blocks = one_shot(d >> 9, (kBlock / 64) * tpw);
    // keep rows x tile blocks within the grid cap; the waves stride over the rest
    const int64_t per_row = one_shot_cap() / rows / 8 * 8;
    if (static_cast<int64_t>(tile_blocks) > per_row)
        tile_blocks = static_cast<unsigned>(per_row < 8 ? 8 : per_row);
    dim3 grid(tile_blocks, static_cast<unsigned>(rows));
    uint8_t* out = reinterpret_cast<uint8_t*>(codes);
    // codes beyond twice the 256 MB Infinity Cache are stored nontemporally
    const int32_t nt_codes = static_cast<int64_t>(rows) * ((d * bits + 7) / 8) > kCodesNontemporalBytes ? 1 : 0;
#define UQ_LAUNCH_QUANTISE(MULTI, BITS)                                                                          \
    do {                                                                                                           \
        if (nt_codes)                                                                                              \
            hipLaunchKernelGGL((k_quantise<MULTI, BITS, true>), grid, dim3(kBlock), 0, stream, g, d, ldg, worker0, \
                               w, S, idx, key0, key1, out, ldc, tpw);                                               \
        else                                                                                                       \
            hipLaunchKernelGGL((k_quantise<MULTI, BITS, false>), grid, dim3(kBlock), 0, stream, g, d, ldg, worker0,\
                               w, S, idx, key0, key1, out, ldc, tpw);                                               \
    } while (0)
    const bool multi = S.K > 1;
    if (bits == 8) {
        if (multi) UQ_LAUNCH_QUANTISE(true, 8); else UQ_LAUNCH_QUANTISE(false, 8);
    } else if (bits == 4) {
        if (multi) UQ_LAUNCH_QUANTISE(true, 4); else UQ_LAUNCH_QUANTISE(false, 4);
    } else {
        if (multi) UQ_LAUNCH_QUANTISE(true, 2); else UQ_LAUNCH_QUANTISE(false, 2);
    }
#undef UQ_LAUNCH_QUANTISE
    return hipGetLastError();
}

hipError_t launch_quant_sum(const float* g, int64_t d, int32_t rows, int64_t ldg, int32_t worker0, const float* w,
                            const ScaleSet& S, const uint8_t* idx, uint64_t seed, int32_t accumulate, int32_t* sum,
                            int32_t M, float* out, hipStream_t stream, int32_t idx_bits)
{
    const bool nib = idx_bits == 4;
    if (d == 0)
        return hipSuccess;
    const uint32_t key0 = static_cast<uint32_t>(seed);
    const uint32_t key1 = static_cast<uint32_t>(seed >> 32);
    // one wave per 512-coordinate tile (at least one block for the tail)
    const dim3 grid(one_shot(d >> 9, kBlock / 64));
    // sums beyond 64 MiB are loaded and stored nontemporally, as in the fused sum
    const bool nt = 4 * d > kSumNontemporalBytes;
    const bool multi = S.K > 1;
    const bool acc = accumulate != 0;
    const bool deq = out != nullptr;
    if (!multi && !acc && deq && rows > 4 && rows <= kFuseRows) {
        // one scale, 5 to 16 rows set and reconstructed: the rows of a tile
        // split over the block's waves, one block per tile
        const dim3 sgrid(one_shot(d >> 9, 1));
#define UQ_LAUNCH_SPLIT(RPW, NT)                                                                                  \
    hipLaunchKernelGGL((k_quant_sum_split<RPW, NT>), sgrid, dim3(kBlock), 0, stream, g, d, rows, ldg, worker0, w,   \
                       S, key0, key1, sum, M, out)
        if (rows <= 8) {
            if (nt)
                UQ_LAUNCH_SPLIT(2, true);
            else
                UQ_LAUNCH_SPLIT(2, false);
        } else {
            if (nt)
                UQ_LAUNCH_SPLIT(4, true);
            else
                UQ_LAUNCH_SPLIT(4, false);
        }
#undef UQ_LAUNCH_SPLIT
        return hipGetLastError();
    }
#define UQ_LAUNCH_QSUM_(MULTI, ACC, DEQ, NT, NIB)                                                                   \
    do {                                                                                                           \
        if (rows == 1)                                                                                             \
            hipLaunchKernelGGL((k_quant_sum<MULTI, ACC, DEQ, NT, true, NIB>), grid, dim3(kBlock), 0, stream, g, d,  \
                               rows, ldg, worker0, w, S, idx, key0, key1, sum, M, out);                            \
        else                                                                                                       \
            hipLaunchKernelGGL((k_quant_sum<MULTI, ACC, DEQ, NT, false, NIB>), grid, dim3(kBlock), 0, stream, g, d, \
                               rows, ldg, worker0, w, S, idx, key0, key1, sum, M, out);                            \
    } while (0)
    // the 4-bit index layout only matters with several scales (NIB = MULTI
    // there, so one scale compiles no second instance)
#define UQ_LAUNCH_QSUM(MULTI, ACC, DEQ, NT)                  \
    do {                                                     \
        if (nib)                                             \
            UQ_LAUNCH_QSUM_(MULTI, ACC, DEQ, NT, MULTI);     \
        else                                                 \
            UQ_LAUNCH_QSUM_(MULTI, ACC, DEQ, NT, false);     \
    } while (0)
#define UQ_LAUNCH_QSUM_NT(MULTI, ACC, DEQ)  \
    do {                                    \
        if (nt)                             \
            UQ_LAUNCH_QSUM(MULTI, ACC, DEQ, true);  \
        else                                \
            UQ_LAUNCH_QSUM(MULTI, ACC, DEQ, false); \
    } while (0)
#define UQ_LAUNCH_QSUM_DEQ(MULTI, ACC)           \
    do {                                         \
        if (deq)                                 \
            UQ_LAUNCH_QSUM_NT(MULTI, ACC, true); \
        else                                     \
            UQ_LAUNCH_QSUM_NT(MULTI, ACC, false);\
    } while (0)
    if (multi) {
        if (acc) UQ_LAUNCH_QSUM_DEQ(true, true); else UQ_LAUNCH_QSUM_DEQ(true, false);
    } else {
        if (acc) UQ_LAUNCH_QSUM_DEQ(false, true); else UQ_LAUNCH_QSUM_DEQ(false, false);
    }
#undef UQ_LAUNCH_QSUM_DEQ
#undef UQ_LAUNCH_QSUM_NT
#undef UQ_LAUNCH_QSUM
#undef UQ_LAUNCH_QSUM_
    return hipGetLastError();
}

hipError_t launch_index_quant_sum(const float* g, int64_t d, int32_t M, int64_t ldg, const float* w,
                                  const ScaleSet& S, uint64_t seed, uint8_t* idx, int32_t* sum, float* out,
                                  hipStream_t stream)
{
    if (d == 0)
        return hipSuccess;
    const uint32_t key0 = static_cast<uint32_t>(seed);
    const uint32_t key1 = static_cast<uint32_t>(seed >> 32);
    const dim3 grid(one_shot(d >> 9, kBlock / 64));
    const bool nt = 4 * d > kSumNontemporalBytes;
#define UQ_LAUNCH_IQS(ROWS)                                                                                        \
    do {                                                                                                           \
        if (nt)                                                                                                    \
            hipLaunchKernelGGL((k_index_quant_sum<ROWS, true>), grid, dim3(kBlock), 0, stream, g, d, M, ldg, w, S, \
                               key0, key1, idx, sum, out);                                                         \
        else                                                                                                       \
            hipLaunchKernelGGL((k_index_quant_sum<ROWS, false>), grid, dim3(kBlock), 0, stream, g, d, M, ldg, w,   \
                               S, key0, key1, idx, sum, out);                                                      \
    } while (0)
    if (M <= 2)
        UQ_LAUNCH_IQS(2);
    else if (M <= 4)
        UQ_LAUNCH_IQS(4);
    else if (M <= 8)
        UQ_LAUNCH_IQS(8);
    else
        UQ_LAUNCH_IQS(16);
#undef UQ_LAUNCH_IQS
    return hipGetLastError();
}

hipError_t launch_index_quantise(const float* g, int64_t d, int32_t M, int64_t ldg, const float* w,
                                 const ScaleSet& S, uint64_t seed, int32_t bits, uint8_t* idx, uint8_t* codes,
                                 int64_t ldc, hipStream_t stream)
{
    if (d == 0)
        return hipSuccess;
    const uint32_t key0 = static_cast<uint32_t>(seed);
    const uint32_t key1 = static_cast<uint32_t>(seed >> 32);
    const dim3 grid(one_shot(d >> 9, kBlock / 64));
    // codes stored nontemporally past the quantiser's threshold, the index with them
    const bool nt = static_cast<int64_t>(M) * ((d * bits + 7) / 8) > kCodesNontemporalBytes;
#define UQ_LAUNCH_IQ_(ROWS, BITS, NT)                                                                             \
    hipLaunchKernelGGL((k_index_quantise<ROWS, BITS, NT>), grid, dim3(kBlock), 0, stream, g, d, M, ldg, w, S, key0, \
                       key1, idx, codes, ldc)
#define UQ_LAUNCH_IQ_B(ROWS, NT)              \
    do {                                      \
        if (bits == 8)                        \
            UQ_LAUNCH_IQ_(ROWS, 8, NT);       \
        else if (bits == 4)                   \
            UQ_LAUNCH_IQ_(ROWS, 4, NT);       \
        else                                  \
            UQ_LAUNCH_IQ_(ROWS, 2, NT);       \
    } while (0)
#define UQ_LAUNCH_IQ(ROWS)                   \
    do {                                     \
        if (nt)                              \
            UQ_LAUNCH_IQ_B(ROWS, true);      \
        else                                 \
            UQ_LAUNCH_IQ_B(ROWS, false);     \
    } while (0)
    if (M <= 2)
        UQ_LAUNCH_IQ(2);
    else if (M <= 4)
        UQ_LAUNCH_IQ(4);
    else if (M <= 8)
        UQ_LAUNCH_IQ(8);
    else
        UQ_LAUNCH_IQ(16);
#undef UQ_LAUNCH_IQ
#undef UQ_LAUNCH_IQ_B
#undef UQ_LAUNCH_IQ_
    return hipGetLastError();
}

hipError_t launch_sum(const int8_t* codes, int64_t d, int32_t rows, int64_t ldc, int32_t accumulate,
                      int32_t* sum, hipStream_t stream)
{
    if (d == 0)
        return hipSuccess;
    const unsigned gx = one_shot(d, kSumTile);
    hipLaunchKernelGGL((k_sum<8, 0>), dim3(gx), dim3(kBlock), 0, stream, reinterpret_cast<const uint8_t*>(codes),
                       d, rows, ldc, accumulate, sum, DeqArgs{});
    return hipGetLastError();
}

hipError_t launch_sum_packed(const uint8_t* packed, int64_t d, int32_t rows, int64_t ldp, int32_t bits,
                             int32_t accumulate, int32_t* sum, hipStream_t stream)
{
    if (d == 0)
        return hipSuccess;
    const unsigned gx = one_shot(d, kSumTile);
    if (bits == 4)
        hipLaunchKernelGGL((k_sum<4, 0>), dim3(gx), dim3(kBlock), 0, stream, packed, d, rows, ldp, accumulate, sum,
                           DeqArgs{});
    else
        hipLaunchKernelGGL((k_sum<2, 0>), dim3(gx), dim3(kBlock), 0, stream, packed, d, rows, ldp, accumulate, sum,
                           DeqArgs{});
    return hipGetLastError();
}

hipError_t launch_sum_dequant(const uint8_t* codes, int64_t d, int32_t rows, int64_t ldc, int32_t bits,
                              int32_t accumulate, int32_t* sum, int32_t M, const float* w, const ScaleSet& S,
                              const uint8_t* idx, float* out, hipStream_t stream)
{
    if (d == 0)
        return hipSuccess;
    const unsigned gx = one_shot(d, kSumTile);
    const DeqArgs da{w, idx, out, S, M, 4 * d > kSumNontemporalBytes ? 1 : 0};
#define UQ_LAUNCH_SUM_DEQ(BITS, DEQ)                                                                               \
    hipLaunchKernelGGL((k_sum<BITS, DEQ>), dim3(gx), dim3(kBlock), 0, stream, codes, d, rows, ldc, accumulate, sum, \
                       da)
    const bool multi = S.K > 1;
    if (bits == 8) {
        if (multi) UQ_LAUNCH_SUM_DEQ(8, 2); else UQ_LAUNCH_SUM_DEQ(8, 1);
    } else if (bits == 4) {
        if (multi) UQ_LAUNCH_SUM_DEQ(4, 2); else UQ_LAUNCH_SUM_DEQ(4, 1);
    } else {
        if (multi) UQ_LAUNCH_SUM_DEQ(2, 2); else UQ_LAUNCH_SUM_DEQ(2, 1);
    }
#undef UQ_LAUNCH_SUM_DEQ
    return hipGetLastError();
}

hipError_t launch_dequant(const int32_t* sum, int64_t d, int32_t M, const float* w, const ScaleSet& S,
                          const uint8_t* idx, float* out, hipStream_t stream)
{
    if (d == 0)
        return hipSuccess;
    const unsigned gx = one_shot((d + 3) / 4, kBlock);
    if (S.K > 1)
        hipLaunchKernelGGL(k_dequant<true>, dim3(gx), dim3(kBlock), 0, stream, sum, d, M, w, S, idx, out);
    else
        hipLaunchKernelGGL(k_dequant<false>, dim3(gx), dim3(kBlock), 0, stream, sum, d, M, w, S, idx, out);
    return hipGetLastError();
}

}  // namespace uq
