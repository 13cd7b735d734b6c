// Device-side building blocks of libuq (gfx950, wave64).
//
// Everything here follows the arithmetic contract in include/uq.h: IEEE
// binary32 products with no contraction (the library is compiled with
// -ffp-contract=off), correctly rounded tables formed in binary64, and the
// Philox4x32-10 counter-based generator of Salmon, Moraes, Dror and Shaw
// ("Parallel random numbers: as easy as 1, 2, 3", SC'11).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace uq {

constexpr int kBlock = 256;          // threads per block: four wave64s
constexpr int kMaxScales = 16;
constexpr float kFloatMax = 3.40282346638528859812e+38f;

// Native clang vectors (HIP's float4 is a wrapper struct, which the
// nontemporal builtins do not accept).
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef int32_t i32x4 __attribute__((ext_vector_type(4)));

// Single-use streams: loads and stores marked nontemporal so they do not
// displace reused lines from the caches.
__device__ __forceinline__ f32x4 load_nt(const float* p)
{
    return __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p));
}
__device__ __forceinline__ i32x4 load_nt(const int32_t* p)
{
    return __builtin_nontemporal_load(reinterpret_cast<const i32x4*>(p));
}
__device__ __forceinline__ uint32_t load_nt_u32(const void* p)
{
    return __builtin_nontemporal_load(reinterpret_cast<const uint32_t*>(p));
}
__device__ __forceinline__ void store_nt(float* p, f32x4 v)
{
    __builtin_nontemporal_store(v, reinterpret_cast<f32x4*>(p));
}

// Scale set passed by value in the kernel arguments.
struct ScaleSet {
    float s[kMaxScales];
    int32_t K;
};

// Philox4x32-10 block function: ten rounds, each multiplying counter words 0
// and 2 by the Philox multipliers (32x32 -> 64 bit), xoring the high halves
// into the other two words together with the round key, and permuting; the
// key advances by the Weyl increments after every round.  The three-way xors
// are single v_bitop3_b32 instructions (truth table 0x96 = a ^ b ^ c).
__device__ __forceinline__ uint4 philox4x32_10(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3,
                                               uint32_t k0, uint32_t k1)
{
#pragma unroll
    for (int round = 0; round < 10; ++round) {
        const uint64_t pa = static_cast<uint64_t>(0xD2511F53u) * c0;
        const uint64_t pb = static_cast<uint64_t>(0xCD9E8D57u) * c2;
        const uint32_t n0 = __builtin_amdgcn_bitop3_b32(static_cast<uint32_t>(pb >> 32), c1, k0, 0x96);
        const uint32_t n2 = __builtin_amdgcn_bitop3_b32(static_cast<uint32_t>(pa >> 32), c3, k1, 0x96);
        c1 = static_cast<uint32_t>(pb);
        c3 = static_cast<uint32_t>(pa);
        c0 = n0;
        c2 = n2;
        k0 += 0x9E3779B9u;
        k1 += 0xBB67AE85u;
    }
    return make_uint4(c0, c1, c2, c3);
}

// RN32(a / b) for binary32 a, b: the binary64 quotient rounded once more to
// binary32 is the correctly rounded binary32 quotient (53 >= 2*24 + 2).
__device__ __forceinline__ float div_rn32(float a, float b)
{
    return static_cast<float>(static_cast<double>(a) / static_cast<double>(b));
}

// The zero path: W not a positive finite binary32, or s_0 / W overflowing.
__device__ __forceinline__ bool zero_path(float W, float inv0)
{
    return !(W > 0.0f) || !(W <= kFloatMax) || !(inv0 <= kFloatMax);
}

// v_cmp_class mask for finite nonzero values (+-normal, +-denormal).
constexpr int kFiniteNonzero = (1 << 3) | (1 << 4) | (1 << 7) | (1 << 8);

// Stochastic level choice for one coordinate from the high 16 bits of its
// uniform word.  inv is 0 on the zero path, so every code is then 0.
//   x = min(|v| * inv, s0)   (0 for zero / NaN / inf v)
//   l = floor(x), t = floor((x - l) * 2^32), code = sign(v) * (l + [r < t])
// With only r's high half known, [r < t] is decided unless the halves tie
// (hi16 == t >> 16), reported in *tie; *t_out and *l_out let the caller
// finish a tie with r's low half.  Returns the signed code as a float.
__device__ __forceinline__ float quantise_hi(float v, float inv, float s0, uint32_t hi16, bool* tie,
                                             uint32_t* t_out, float* l_out)
{
    const bool ok = __builtin_amdgcn_classf(v, kFiniteNonzero);
    float x = fabsf(v) * inv;
    x = ok ? x : 0.0f;
    x = fminf(x, s0);
    const float lf = floorf(x);
    const uint32_t t = static_cast<uint32_t>((x - lf) * 4294967296.0f);
    const uint32_t th = t >> 16;
    *tie = hi16 == th;
    *t_out = t;
    *l_out = lf;
    const float mag = lf + (hi16 < th ? 1.0f : 0.0f);
    return copysignf(mag, v);
}

__device__ __forceinline__ uint32_t pack4(int32_t a, int32_t b, int32_t c, int32_t d)
{
    return (static_cast<uint32_t>(a) & 0xFFu) | ((static_cast<uint32_t>(b) & 0xFFu) << 8) |
           ((static_cast<uint32_t>(c) & 0xFFu) << 16) | (static_cast<uint32_t>(d) << 24);
}

// Deterministic wave64 sum of a double (fixed butterfly order).
__device__ __forceinline__ double wave_sum(double x)
{
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1)
        x += __shfl_xor(x, off, 64);
    return x;
}

}  // namespace uq
