// Achievable-bandwidth references for reading the hot path's rooflines:
// streaming kernels with the access patterns of the hot path and no work.
// Built into their own library (libuq_probe.so); the quantiser library does
// not contain or call them.
//
//   uqp_read           : n fp32 read with 16-byte nontemporal loads by a
//                        grid-stride loop over 8192 blocks (the best of a
//                        sweep of grid sizes for a pure read); one float per
//                        thread written out.
//   uqp_read_write8    : n fp32 read in 512-element wave tiles (16-byte loads
//                        per lane, two per tile) and one byte written per
//                        element (the quantiser's pattern); the byte is the
//                        float's top byte.
//   uqp_rows_read      : the first d fp32 of each of M rows (row stride ldg)
//                        read by blocks of one 65536-element chunk of one row
//                        (the norm pass's bytes, 4 M per coordinate, as a
//                        pure read); one float per block written out.
//   uqp_accumulate     : the fused quantise-and-sum's bytes for one streamed
//                        worker with no work: per element 4 bytes of g, 1 of
//                        idx and 4 of sum read, 4 of sum written, in the same
//                        512-element wave tiles; sum[i] += idx[i] + (int)g[i].
//   uqp_copy           : n fp32 copied (16-byte nontemporal loads and stores).
//   uqp_keys_index     : the index pass's bytes with no work: d 16-bit keys
//                        read (16-byte nontemporal loads, one octet of keys
//                        per load) and d bytes written (8-byte nontemporal
//                        stores, the low byte of each key); a block covers
//                        256 * octs octets, thread t octets t, t + 256, ...
// n (d for the row and accumulate probes) must be a multiple of 512; every
// pointer 16-byte aligned; out holds uqp_read_out_floats(n) floats
// (uqp_rows_read: uqp_rows_out_floats(d, M)).  Returns 0, or -1 on a bad
// argument / -5 on a launch failure.
#include <hip/hip_runtime.h>

#include <cstdint>

namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
constexpr int kBlock = 256;
constexpr int64_t kMaxBlocks = int64_t(1) << 22;

__device__ __forceinline__ f32x4 ld(const float* p)
{
    return __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p));
}

__global__ __launch_bounds__(kBlock) void k_read(const float* __restrict__ g, int64_t nquad,
                                                 float* __restrict__ out)
{
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock;
    float s = 0.0f;
    for (int64_t q = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; q < nquad; q += stride) {
        const f32x4 v = ld(g + (q << 2));
        s += v.x + v.y + v.z + v.w;
    }
    out[static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x] = s;
}

__global__ __launch_bounds__(kBlock) void k_read_write8(const float* __restrict__ g, int64_t ntiles,
                                                        uint8_t* __restrict__ c)
{
    const int lane = threadIdx.x & 63;
    const int64_t nwaves = static_cast<int64_t>(gridDim.x) * (kBlock / 64);
    for (int64_t T = static_cast<int64_t>(blockIdx.x) * (kBlock / 64) + (threadIdx.x >> 6); T < ntiles;
         T += nwaves) {
        const int64_t a = (T << 9) + 4 * lane;
        const f32x4 A = ld(g + a);
        const f32x4 B = ld(g + a + 256);
        const uint32_t wa = __builtin_amdgcn_perm(
            __builtin_amdgcn_perm(__float_as_uint(A.w), __float_as_uint(A.z), 0x0703u),
            __builtin_amdgcn_perm(__float_as_uint(A.y), __float_as_uint(A.x), 0x0703u), 0x05040100u);
        const uint32_t wb = __builtin_amdgcn_perm(
            __builtin_amdgcn_perm(__float_as_uint(B.w), __float_as_uint(B.z), 0x0703u),
            __builtin_amdgcn_perm(__float_as_uint(B.y), __float_as_uint(B.x), 0x0703u), 0x05040100u);
        *reinterpret_cast<uint32_t*>(c + a) = wa;
        *reinterpret_cast<uint32_t*>(c + a + 256) = wb;
    }
}

constexpr int64_t kRowChunk = 65536;

__global__ __launch_bounds__(kBlock) void k_rows_read(const float* __restrict__ g, int64_t d, int64_t ldg,
                                                      int64_t nchunks, float* __restrict__ out)
{
    const int64_t c = blockIdx.x;
    const int64_t begin = c * kRowChunk;
    const int64_t end = begin + kRowChunk < d ? begin + kRowChunk : d;
    const float* row = g + static_cast<int64_t>(blockIdx.y) * ldg;
    float s = 0.0f;
    for (int64_t q = (begin >> 2) + threadIdx.x; q < (end >> 2); q += kBlock) {
        const f32x4 v = ld(row + (q << 2));
        s += v.x + v.y + v.z + v.w;
    }
    // block sum in a fixed order
    __shared__ float part[kBlock];
    part[threadIdx.x] = s;
    __syncthreads();
    if (threadIdx.x == 0) {
        float t = 0.0f;
        for (int i = 0; i < kBlock; ++i)
            t += part[i];
        out[static_cast<int64_t>(blockIdx.y) * nchunks + c] = t;
    }
}

typedef int32_t i32x4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(kBlock) void k_accumulate(const float* __restrict__ g, const uint8_t* __restrict__ idx,
                                                       int32_t* __restrict__ sum, int64_t ntiles)
{
    const int lane = threadIdx.x & 63;
    const int64_t T = static_cast<int64_t>(blockIdx.x) * (kBlock / 64) + (threadIdx.x >> 6);
    if (T >= ntiles)
        return;
    const int64_t a = (T << 9) + 4 * lane;
    const f32x4 A = ld(g + a), B = ld(g + a + 256);
    const uint32_t ka = *reinterpret_cast<const uint32_t*>(idx + a);
    const uint32_t kb = *reinterpret_cast<const uint32_t*>(idx + a + 256);
    i32x4 sa = __builtin_nontemporal_load(reinterpret_cast<const i32x4*>(sum + a));
    i32x4 sb = __builtin_nontemporal_load(reinterpret_cast<const i32x4*>(sum + a + 256));
    sa.x += static_cast<int32_t>(ka & 0xFFu) + static_cast<int32_t>(A.x);
    sa.y += static_cast<int32_t>((ka >> 8) & 0xFFu) + static_cast<int32_t>(A.y);
    sa.z += static_cast<int32_t>((ka >> 16) & 0xFFu) + static_cast<int32_t>(A.z);
    sa.w += static_cast<int32_t>(ka >> 24) + static_cast<int32_t>(A.w);
    sb.x += static_cast<int32_t>(kb & 0xFFu) + static_cast<int32_t>(B.x);
    sb.y += static_cast<int32_t>((kb >> 8) & 0xFFu) + static_cast<int32_t>(B.y);
    sb.z += static_cast<int32_t>((kb >> 16) & 0xFFu) + static_cast<int32_t>(B.z);
    sb.w += static_cast<int32_t>(kb >> 24) + static_cast<int32_t>(B.w);
    __builtin_nontemporal_store(sa, reinterpret_cast<i32x4*>(sum + a));
    __builtin_nontemporal_store(sb, reinterpret_cast<i32x4*>(sum + a + 256));
}

__global__ __launch_bounds__(kBlock) void k_copy(const float* __restrict__ src, float* __restrict__ dst, int64_t nquad)
{
    const int64_t q = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
    if (q < nquad)
        __builtin_nontemporal_store(ld(src + (q << 2)), reinterpret_cast<f32x4*>(dst + (q << 2)));
}

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

template <int OCTS>
__global__ __launch_bounds__(kBlock) void k_keys_index(const uint16_t* __restrict__ keys, uint8_t* __restrict__ idx,
                                                       int64_t noct)
{
    const int64_t o0 = static_cast<int64_t>(blockIdx.x) * (kBlock * OCTS) + threadIdx.x;
    u32x4 kv[OCTS];
#pragma unroll
    for (int j = 0; j < OCTS; ++j) {
        const int64_t o = o0 + kBlock * j;
        kv[j] = o < noct ? __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(keys + (o << 3)))
                         : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int j = 0; j < OCTS; ++j) {
        const int64_t o = o0 + kBlock * j;
        if (o < noct) {
            u32x2 b;
            b.x = __builtin_amdgcn_perm(kv[j].y, kv[j].x, 0x06040200u);
            b.y = __builtin_amdgcn_perm(kv[j].w, kv[j].z, 0x06040200u);
            __builtin_nontemporal_store(b, reinterpret_cast<u32x2*>(idx + (o << 3)));
        }
    }
}

int64_t blocks_for(int64_t units, int64_t per_block)
{
    const int64_t b = (units + per_block - 1) / per_block;
    return b < 1 ? 1 : (b > kMaxBlocks ? kMaxBlocks : b);
}

bool ok_args(const void* g, int64_t n, const void* out)
{
    return g != nullptr && out != nullptr && n > 0 && n % 512 == 0 &&
           reinterpret_cast<uintptr_t>(g) % 16 == 0 && reinterpret_cast<uintptr_t>(out) % 16 == 0;
}

}  // namespace

extern "C" {

constexpr int64_t kReadBlocks = 8192;

int64_t uqp_read_out_floats(int64_t n)
{
    const int64_t b = blocks_for(n / 4, kBlock);
    return (b < kReadBlocks ? b : kReadBlocks) * kBlock;
}

int uqp_read(const float* g, int64_t n, float* out, void* stream)
{
    if (!ok_args(g, n, out))
        return -1;
    const int64_t b = blocks_for(n / 4, kBlock);
    const int64_t blocks = b < kReadBlocks ? b : kReadBlocks;
    hipLaunchKernelGGL(k_read, dim3(static_cast<unsigned>(blocks)), dim3(kBlock), 0,
                       static_cast<hipStream_t>(stream), g, n / 4, out);
    return hipGetLastError() == hipSuccess ? 0 : -5;
}

int uqp_read_write8(const float* g, int64_t n, uint8_t* c, void* stream)
{
    if (!ok_args(g, n, c))
        return -1;
    const int64_t blocks = blocks_for(n / 512, kBlock / 64);
    hipLaunchKernelGGL(k_read_write8, dim3(static_cast<unsigned>(blocks)), dim3(kBlock), 0,
                       static_cast<hipStream_t>(stream), g, n / 512, c);
    return hipGetLastError() == hipSuccess ? 0 : -5;
}

int64_t uqp_rows_out_floats(int64_t d, int32_t M)
{
    return (d + kRowChunk - 1) / kRowChunk * (M > 0 ? M : 0);
}

int uqp_rows_read(const float* g, int64_t d, int32_t M, int64_t ldg, float* out, void* stream)
{
    if (!ok_args(g, d, out) || M < 1 || M > 65535 || ldg < d || ldg % 4 != 0)
        return -1;
    const int64_t nchunks = (d + kRowChunk - 1) / kRowChunk;
    if (nchunks > kMaxBlocks)
        return -1;
    hipLaunchKernelGGL(k_rows_read, dim3(static_cast<unsigned>(nchunks), static_cast<unsigned>(M)), dim3(kBlock), 0,
                       static_cast<hipStream_t>(stream), g, d, ldg, nchunks, out);
    return hipGetLastError() == hipSuccess ? 0 : -5;
}

int uqp_accumulate(const float* g, const uint8_t* idx, int32_t* sum, int64_t d, void* stream)
{
    if (!ok_args(g, d, sum) || idx == nullptr || reinterpret_cast<uintptr_t>(idx) % 16 != 0)
        return -1;
    const int64_t ntiles = d / 512;
    const int64_t blocks = (ntiles + kBlock / 64 - 1) / (kBlock / 64);
    if (blocks > kMaxBlocks)
        return -1;
    hipLaunchKernelGGL(k_accumulate, dim3(static_cast<unsigned>(blocks)), dim3(kBlock), 0,
                       static_cast<hipStream_t>(stream), g, idx, sum, ntiles);
    return hipGetLastError() == hipSuccess ? 0 : -5;
}

int uqp_copy(const float* src, float* dst, int64_t n, void* stream)
{
    if (!ok_args(src, n, dst))
        return -1;
    const int64_t blocks = blocks_for(n / 4, kBlock);
    if ((n / 4 + kBlock - 1) / kBlock > kMaxBlocks)
        return -1;
    hipLaunchKernelGGL(k_copy, dim3(static_cast<unsigned>(blocks)), dim3(kBlock), 0,
                       static_cast<hipStream_t>(stream), src, dst, n / 4);
    return hipGetLastError() == hipSuccess ? 0 : -5;
}

int uqp_keys_index(const uint16_t* keys, int64_t d, uint8_t* idx, int32_t octs, void* stream)
{
    if (!ok_args(keys, d, idx) || (octs != 2 && octs != 4 && octs != 8))
        return -1;
    const int64_t noct = d / 8;
    const int64_t blocks = (noct + kBlock * octs - 1) / (kBlock * octs);
    if (blocks > kMaxBlocks)
        return -1;
    const hipStream_t s = static_cast<hipStream_t>(stream);
    if (octs == 2)
        hipLaunchKernelGGL(k_keys_index<2>, dim3(static_cast<unsigned>(blocks)), dim3(kBlock), 0, s, keys, idx, noct);
    else if (octs == 4)
        hipLaunchKernelGGL(k_keys_index<4>, dim3(static_cast<unsigned>(blocks)), dim3(kBlock), 0, s, keys, idx, noct);
    else
        hipLaunchKernelGGL(k_keys_index<8>, dim3(static_cast<unsigned>(blocks)), dim3(kBlock), 0, s, keys, idx, noct);
    return hipGetLastError() == hipSuccess ? 0 : -5;
}

}  // extern "C"
