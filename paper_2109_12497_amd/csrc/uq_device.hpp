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
typedef uint16_t u16x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

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
__device__ __forceinline__ u32x4 load_nt(const uint32_t* p)
{
    return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
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
    float s_last;  // s[K - 1]
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

// v_cmp_class masks: finite nonzero values (+-normal, +-denormal); NaN and
// infinities.
constexpr int kFiniteNonzero = (1 << 3) | (1 << 4) | (1 << 7) | (1 << 8);
constexpr int kNonFinite = (1 << 0) | (1 << 1) | (1 << 2) | (1 << 9);

// sign(v) * mag for an integer magnitude (v's sign bit; 0 stays 0).
__device__ __forceinline__ int32_t apply_sign(uint32_t mag, float v)
{
    const int32_t s = __float_as_int(v) >> 31;
    return (static_cast<int32_t>(mag) ^ s) - s;
}

// x = min(|v| * inv, s0), 0 for zero / NaN / inf v.  inv is 0 on the zero
// path, so every code is then 0.
__device__ __forceinline__ float scaled_magnitude(float v, float inv, float s0)
{
    const bool ok = __builtin_amdgcn_classf(v, kFiniteNonzero);
    const float x = fabsf(v) * inv;
    return fminf(ok ? x : 0.0f, s0);
}

// Stochastic level choice for one coordinate from the high 16 bits of its
// uniform word:
//   l = floor(x), t = floor((x - l) * 2^32), code = sign(v) * (l + [r < t])
// As 0 <= x <= 127, T = floor(x * 2^16) is exact and equals
// l * 2^16 + (t >> 16): one conversion yields the level and the high half of
// the threshold.  With only r's high half known, [r < t] is decided unless
// the halves tie (hi16 == t >> 16), reported in *tie; the caller finishes a
// tie from x (*x_out) and r's low half with quantise_tie.
__device__ __forceinline__ int32_t quantise_hi(float v, float inv, float s0, uint32_t hi16, bool* tie,
                                               float* x_out)
{
    const float x = scaled_magnitude(v, inv, s0);
    const uint32_t T = static_cast<uint32_t>(x * 65536.0f);
    const uint32_t th = T & 0xFFFFu;
    *tie = hi16 == th;
    *x_out = x;
    return apply_sign((T >> 16) + (hi16 < th ? 1u : 0u), v);
}

// The same decision for two coordinates at once in the 16-bit lanes of one
// register (packed integer ops): T0, T1 as above, r01 their high random
// halves (coordinate 0 in the low lane).  Returns the two codes as 16-bit
// two's complement lanes.  one2 holds 1 in both lanes; it is passed in so
// that the packed min is not rewritten as two compares and selects.
__device__ __forceinline__ uint32_t pair_codes(uint32_t T0, uint32_t T1, float v0, float v1, uint32_t r01,
                                               uint32_t one2)
{
    const u16x2 lev = __builtin_bit_cast(u16x2, __builtin_amdgcn_perm(T1, T0, 0x07060302u));
    const u16x2 th = __builtin_bit_cast(u16x2, __builtin_amdgcn_perm(T1, T0, 0x05040100u));
    // max(th - r, 0) > 0 exactly when r < th
    const u16x2 up = __builtin_elementwise_min(__builtin_elementwise_sub_sat(th, __builtin_bit_cast(u16x2, r01)),
                                               __builtin_bit_cast(u16x2, one2));
    const u16x2 mag = lev + up;
    // 0xFFFF in the lane of a negative v (replicated sign bits of the top bytes)
    const u16x2 neg = __builtin_bit_cast(
        u16x2, __builtin_amdgcn_perm(__float_as_uint(v1), __float_as_uint(v0), 0x0B0B0909u));
    return __builtin_bit_cast(uint32_t, static_cast<u16x2>((mag ^ neg) - neg));
}

// The tied case: [r < t] decided by the low halves of r and t.
__device__ __forceinline__ int32_t quantise_tie(float v, float x, uint32_t lo16)
{
    const float lf = floorf(x);
    const uint32_t t = static_cast<uint32_t>((x - lf) * 4294967296.0f);
    return apply_sign(static_cast<uint32_t>(lf) + (lo16 < (t & 0xFFFFu) ? 1u : 0u), v);
}

// The tied case from xs = x * 2^16 and T = floor(xs): the low half of t is
// floor((xs - T) * 2^16).
__device__ __forceinline__ int32_t quantise_tie_scaled(float v, float xs, uint32_t T, uint32_t lo16)
{
    const uint32_t t_lo = static_cast<uint32_t>((xs - floorf(xs)) * 65536.0f);
    return apply_sign((T >> 16) + (lo16 < t_lo ? 1u : 0u), v);
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
