// Achievable-bandwidth references for reading the quantiser's roofline: two
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
// n must be a multiple of 512; g and c 16-byte aligned; out holds
// uqp_read_out_floats(n) floats.  Returns 0, or -1 on a bad argument / -5 on a
// launch failure.
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

}  // extern "C"
