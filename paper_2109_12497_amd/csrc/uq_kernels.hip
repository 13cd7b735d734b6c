// HIP kernels of libuq for MI355X (gfx950).
//
// The aggregation step of Algorithm 1 / Algorithm 2 (Sec. 3.1-3.2) runs as
// five streaming kernels, each bound by HBM bandwidth:
//   k_sumsq     per-row, per-chunk fp64 sums of squares        (norm, pass 1)
//   k_finish    fixed-order reduction of the chunk sums, max    (norm, pass 2)
//               over rows, sqrt -> W
//   k_index     shared scale index from the largest |g| over    (Eq. (11) +
//               the workers at each coordinate                    sharing)
//   k_quantise  Philox draws + stochastic rounding + int8 pack  (Eq. (8)/(12))
//   k_sum       int8 rows -> int32                               (all-reduce)
//   k_dequant   int32 (+ index) -> fp32                          (Eq. (9)/(13))
//
// Every per-coordinate result is a pure function of its inputs and the
// coordinate index, so the output is independent of the launch geometry;
// the norm's reduction tree depends only on d.
#include "uq_device.hpp"
#include "uq_launch.hpp"

namespace uq {

// ---------------------------------------------------------------------------
// Norm, pass 1: block (c, m) sums g[m][c*chunk .. min(d, (c+1)*chunk)) squared
// in binary64 (each square exact) and stores the partial in part[m*nchunks+c].
// chunk is a multiple of 1024, so every chunk starts 16-byte aligned.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kBlock) void k_sumsq(const float* __restrict__ g, int64_t d, int64_t ldg,
                                                  int64_t chunk, int32_t nchunks,
                                                  double* __restrict__ part)
{
    const int32_t c = blockIdx.x;
    const int32_t m = blockIdx.y;
    const float* row = g + static_cast<int64_t>(m) * ldg;
    const int64_t begin = static_cast<int64_t>(c) * chunk;
    const int64_t end = begin + chunk < d ? begin + chunk : d;
    const int64_t nvec = (end - begin) >> 2;
    const float* v4 = row + begin;

    double acc0 = 0.0, acc1 = 0.0, acc2 = 0.0, acc3 = 0.0;
    int64_t j = threadIdx.x;
    for (; j + 3 * kBlock < nvec; j += 4 * kBlock) {
        const f32x4 a = load_nt(v4 + 4 * (j));
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
        const f32x4 a = load_nt(v4 + 4 * (j));
        acc0 = fma((double)a.x, (double)a.x, acc0); acc1 = fma((double)a.y, (double)a.y, acc1);
        acc2 = fma((double)a.z, (double)a.z, acc2); acc3 = fma((double)a.w, (double)a.w, acc3);
    }
    // at most three trailing coordinates (only in the last chunk when d % 4 != 0)
    const int64_t tail = begin + (nvec << 2) + threadIdx.x;
    if (tail < end) {
        const double x = row[tail];
        acc0 = fma(x, x, acc0);
    }
    double s = wave_sum((acc0 + acc1) + (acc2 + acc3));

    __shared__ double wave_part[kBlock / 64];
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    if (lane == 0)
        wave_part[wave] = s;
    __syncthreads();
    if (threadIdx.x == 0) {
        const double total = (wave_part[0] + wave_part[1]) + (wave_part[2] + wave_part[3]);
        part[static_cast<int64_t>(m) * nchunks + c] = total;
    }
}

// ---------------------------------------------------------------------------
// Norm, pass 2 (one block): S_m = fixed-order sum of row m's chunk partials;
// W = RN32(sqrt(max_m S_m)), NaN if any S_m is NaN.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kBlock) void k_finish(const double* __restrict__ part, int32_t nchunks,
                                                   int32_t M, float* __restrict__ w)
{
    __shared__ double wave_part[kBlock / 64];
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    double best = 0.0;
    bool any_nan = false;
    for (int32_t m = 0; m < M; ++m) {
        const double* p = part + static_cast<int64_t>(m) * nchunks;
        double s = 0.0;
        for (int32_t c = threadIdx.x; c < nchunks; c += kBlock)
            s += p[c];
        s = wave_sum(s);
        if (lane == 0)
            wave_part[wave] = s;
        __syncthreads();
        const double S = (wave_part[0] + wave_part[1]) + (wave_part[2] + wave_part[3]);
        __syncthreads();
        any_nan = any_nan || (S != S);
        best = S > best ? S : best;
    }
    if (threadIdx.x == 0)
        *w = any_nan ? __builtin_nanf("") : static_cast<float>(sqrt(best));
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

__global__ __launch_bounds__(kBlock) void k_index(const float* __restrict__ g, int64_t d, int32_t M,
                                                  int64_t ldg, const float* __restrict__ wptr,
                                                  ScaleSet S, uint8_t* __restrict__ idx)
{
    __shared__ float inv_s[kMaxScales];
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

    const int64_t nquad = d >> 2;
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock;
    for (int64_t q = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; q < nquad; q += stride) {
        float4 amax = make_float4(0.f, 0.f, 0.f, 0.f);
        const float* p = g + (q << 2);
        for (int32_t m = 0; m < M; ++m) {
            const f32x4 v = load_nt(p + static_cast<int64_t>(m) * ldg);
            amax.x = fmaxf(amax.x, usable_or_zero(v.x));
            amax.y = fmaxf(amax.y, usable_or_zero(v.y));
            amax.z = fmaxf(amax.z, usable_or_zero(v.z));
            amax.w = fmaxf(amax.w, usable_or_zero(v.w));
        }
        const uint32_t packed = index_of(amax.x, inv, K, s0, zero) |
                                (index_of(amax.y, inv, K, s0, zero) << 8) |
                                (index_of(amax.z, inv, K, s0, zero) << 16) |
                                (index_of(amax.w, inv, K, s0, zero) << 24);
        *reinterpret_cast<uint32_t*>(idx + (q << 2)) = packed;
    }
    // trailing d % 4 coordinates
    const int64_t t = (nquad << 2) + static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
    if (blockIdx.x == 0 && t < d) {
        float amax = 0.0f;
        for (int32_t m = 0; m < M; ++m)
            amax = fmaxf(amax, usable_or_zero(g[static_cast<int64_t>(m) * ldg + t]));
        idx[t] = static_cast<uint8_t>(index_of(amax, inv, K, s0, zero));
    }
}

// ---------------------------------------------------------------------------
// Quantisation.  One thread handles a group of 8 consecutive coordinates,
// which is exactly one Philox block: its eight 16-bit halves are the high
// halves of the coordinates' uniform words.  The low halves (a second block
// with counter word 3 = 1) are drawn only for the rare coordinates whose high
// half equals the threshold's (probability 2^-16 each).
// ---------------------------------------------------------------------------
template <bool MULTI>
__global__ __launch_bounds__(kBlock) void k_quantise(const float* __restrict__ g, int64_t d, int64_t ldg,
                                                     int32_t worker0, const float* __restrict__ wptr,
                                                     ScaleSet S, const uint8_t* __restrict__ idx,
                                                     uint32_t key0, uint32_t key1,
                                                     int8_t* __restrict__ codes, int64_t ldc)
{
    __shared__ float inv_s[kMaxScales];
    const float W = *wptr;
    float inv0;
    if (MULTI) {
        if (threadIdx.x < S.K)
            inv_s[threadIdx.x] = div_rn32(S.s[threadIdx.x], W);
        __syncthreads();
        inv0 = inv_s[0];
    } else {
        inv0 = div_rn32(S.s[0], W);
    }
    const bool zero = zero_path(W, inv0);
    const float s0 = S.s[0];
    const int32_t kmax = S.K - 1;

    const int32_t r = blockIdx.y;
    const uint32_t worker = static_cast<uint32_t>(worker0) + static_cast<uint32_t>(r);
    const float* row = g + static_cast<int64_t>(r) * ldg;
    int8_t* out = codes + static_cast<int64_t>(r) * ldc;

    const int64_t nfull = d >> 3;
    const int64_t ngroups = (d + 7) >> 3;
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock;
    for (int64_t q = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; q < ngroups; q += stride) {
        const int64_t base = q << 3;
        const bool full = q < nfull;
        float v[8];
        float inv[8];
        if (full) {
            const f32x4 a = load_nt(row + base);
            const f32x4 b = load_nt(row + base + 4);
            v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
            v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
        } else {
#pragma unroll
            for (int j = 0; j < 8; ++j)
                v[j] = base + j < d ? row[base + j] : 0.0f;
        }
        if (MULTI) {
            uint8_t k8[8];
            if (full) {
                const uint2 kk = *reinterpret_cast<const uint2*>(idx + base);
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    k8[j] = static_cast<uint8_t>(kk.x >> (8 * j));
                    k8[j + 4] = static_cast<uint8_t>(kk.y >> (8 * j));
                }
            } else {
#pragma unroll
                for (int j = 0; j < 8; ++j)
                    k8[j] = base + j < d ? idx[base + j] : 0;
            }
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const int32_t k = k8[j] < kmax ? k8[j] : kmax;
                inv[j] = inv_s[k];
            }
        } else {
#pragma unroll
            for (int j = 0; j < 8; ++j)
                inv[j] = inv0;
        }

        const uint4 hi = philox4x32_10(static_cast<uint32_t>(q), static_cast<uint32_t>(q >> 32), worker,
                                       0u, key0, key1);
        const uint32_t hw[4] = {hi.x, hi.y, hi.z, hi.w};
        int32_t code[8], level[8];
        uint32_t tlow[8];
        bool tie[8];
        bool any_tie = false;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const uint32_t h16 = j < 4 ? (hw[j] & 0xFFFFu) : (hw[j - 4] >> 16);
            const bool ok = !zero && usable(fabsf(v[j]));
            code[j] = quantise_hi(v[j], inv[j], s0, h16, ok, &tie[j], &tlow[j], &level[j]);
            any_tie = any_tie || tie[j];
        }
        if (any_tie) {
            const uint4 lo = philox4x32_10(static_cast<uint32_t>(q), static_cast<uint32_t>(q >> 32),
                                           worker, 1u, key0, key1);
            const uint32_t lw[4] = {lo.x, lo.y, lo.z, lo.w};
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                if (tie[j]) {
                    const uint32_t l16 = j < 4 ? (lw[j] & 0xFFFFu) : (lw[j - 4] >> 16);
                    const int32_t mag = level[j] + (l16 < tlow[j] ? 1 : 0);
                    code[j] = v[j] < 0.0f ? -mag : mag;
                }
            }
        }
        if (full) {
            uint2 packed;
            packed.x = pack4(code[0], code[1], code[2], code[3]);
            packed.y = pack4(code[4], code[5], code[6], code[7]);
            *reinterpret_cast<uint2*>(out + base) = packed;
        } else {
#pragma unroll
            for (int j = 0; j < 8; ++j)
                if (base + j < d)
                    out[base + j] = static_cast<int8_t>(code[j]);
        }
    }
}

// ---------------------------------------------------------------------------
// Integer sum of the rows' codes (the all-reduce), four coordinates per
// thread per step.
// ---------------------------------------------------------------------------
__device__ __forceinline__ int32_t sbyte(uint32_t w, int j)
{
    return static_cast<int32_t>(static_cast<int8_t>(w >> (8 * j)));
}

__global__ __launch_bounds__(kBlock) void k_sum(const int8_t* __restrict__ codes, int64_t d, int32_t rows,
                                                int64_t ldc, int32_t accumulate, int32_t* __restrict__ sum)
{
    const int64_t nquad = d >> 2;
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock;
    for (int64_t q = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; q < nquad; q += stride) {
        int4 acc = make_int4(0, 0, 0, 0);
        if (accumulate)
            acc = *reinterpret_cast<const int4*>(sum + (q << 2));
        const int8_t* p = codes + (q << 2);
        for (int32_t r = 0; r < rows; ++r) {
            const uint32_t w = load_nt_u32(p + static_cast<int64_t>(r) * ldc);
            acc.x += sbyte(w, 0);
            acc.y += sbyte(w, 1);
            acc.z += sbyte(w, 2);
            acc.w += sbyte(w, 3);
        }
        *reinterpret_cast<int4*>(sum + (q << 2)) = acc;
    }
    const int64_t t = (nquad << 2) + static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
    if (blockIdx.x == 0 && t < d) {
        int32_t acc = accumulate ? sum[t] : 0;
        for (int32_t r = 0; r < rows; ++r)
            acc += codes[static_cast<int64_t>(r) * ldc + t];
        sum[t] = acc;
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

    const int64_t nquad = d >> 2;
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock;
    for (int64_t q = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; q < nquad; q += stride) {
        const i32x4 s = load_nt(sum + (q << 2));
        f32x4 o;
        if (MULTI) {
            const uint32_t kk = *reinterpret_cast<const uint32_t*>(idx + (q << 2));
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
// Host-side launchers (called by the ABI layer after validation).
// ---------------------------------------------------------------------------
static unsigned grid_for(int64_t units, int64_t cap)
{
    int64_t blocks = (units + kBlock - 1) / kBlock;
    if (blocks > cap)
        blocks = cap;
    return static_cast<unsigned>(blocks < 1 ? 1 : blocks);
}

hipError_t launch_shared_scale(const float* g, int64_t d, int32_t M, int64_t ldg, const ScaleSet& S,
                               float* w, uint8_t* idx, double* part, hipStream_t stream)
{
    const NormPlan plan = norm_plan(d);
    if (plan.nchunks > 0) {
        dim3 grid(static_cast<unsigned>(plan.nchunks), static_cast<unsigned>(M));
        hipLaunchKernelGGL(k_sumsq, grid, dim3(kBlock), 0, stream, g, d, ldg, plan.chunk, plan.nchunks, part);
    }
    hipLaunchKernelGGL(k_finish, dim3(1), dim3(kBlock), 0, stream, part, plan.nchunks, M, w);
    if (S.K > 1 && d > 0) {
        const unsigned gx = grid_for((d + 3) / 4, grid_cap());
        hipLaunchKernelGGL(k_index, dim3(gx), dim3(kBlock), 0, stream, g, d, M, ldg, w, S, idx);
    }
    return hipGetLastError();
}

hipError_t launch_quantise(const float* g, int64_t d, int32_t rows, int64_t ldg, int32_t worker0,
                           const float* w, const ScaleSet& S, const uint8_t* idx, uint64_t seed,
                           int8_t* codes, int64_t ldc, hipStream_t stream)
{
    if (d == 0)
        return hipSuccess;
    int64_t cap = grid_cap() / rows;
    if (cap < 1)
        cap = 1;
    const unsigned gx = grid_for((d + 7) / 8, cap);
    const uint32_t key0 = static_cast<uint32_t>(seed);
    const uint32_t key1 = static_cast<uint32_t>(seed >> 32);
    dim3 grid(gx, static_cast<unsigned>(rows));
    if (S.K > 1)
        hipLaunchKernelGGL(k_quantise<true>, grid, dim3(kBlock), 0, stream, g, d, ldg, worker0, w, S, idx,
                           key0, key1, codes, ldc);
    else
        hipLaunchKernelGGL(k_quantise<false>, grid, dim3(kBlock), 0, stream, g, d, ldg, worker0, w, S,
                           idx, key0, key1, codes, ldc);
    return hipGetLastError();
}

hipError_t launch_sum(const int8_t* codes, int64_t d, int32_t rows, int64_t ldc, int32_t accumulate,
                      int32_t* sum, hipStream_t stream)
{
    if (d == 0)
        return hipSuccess;
    const unsigned gx = grid_for((d + 3) / 4, grid_cap());
    hipLaunchKernelGGL(k_sum, dim3(gx), dim3(kBlock), 0, stream, codes, d, rows, ldc, accumulate, sum);
    return hipGetLastError();
}

hipError_t launch_dequant(const int32_t* sum, int64_t d, int32_t M, const float* w, const ScaleSet& S,
                          const uint8_t* idx, float* out, hipStream_t stream)
{
    if (d == 0)
        return hipSuccess;
    const unsigned gx = grid_for((d + 3) / 4, grid_cap());
    if (S.K > 1)
        hipLaunchKernelGGL(k_dequant<true>, dim3(gx), dim3(kBlock), 0, stream, sum, d, M, w, S, idx, out);
    else
        hipLaunchKernelGGL(k_dequant<false>, dim3(gx), dim3(kBlock), 0, stream, sum, d, M, w, S, idx, out);
    return hipGetLastError();
}

}  // namespace uq
