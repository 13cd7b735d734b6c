// Test helper (not part of libuq): runs the library's own device arithmetic
// for the scale tables on arrays, so that a test can compare it bitwise with
// the host's IEEE binary32 operations.
//   uqt_div_rn32(a, b, q, n)   q[i] = div_rn32(a[i], b[i])  (inv_k = s_k / W,
//                                                           deq_k = W / (M s_k))
//   uqt_sqrt_rn32(s, w, n)     w[i] = RN32(sqrt(s[i]))      (W from the fp64
//                                                           sum of squares)
// Device pointers; returns 0, or -1 on a bad argument / -5 on a launch failure.
#include "uq_device.hpp"

namespace {

constexpr int kThreads = 256;

__global__ __launch_bounds__(kThreads) void k_div(const float* __restrict__ a, const float* __restrict__ b,
                                                  float* __restrict__ q, int64_t n)
{
    const int64_t i = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x;
    if (i < n)
        q[i] = uq::div_rn32(a[i], b[i]);
}

__global__ __launch_bounds__(kThreads) void k_sqrt(const double* __restrict__ s, float* __restrict__ w, int64_t n)
{
    const int64_t i = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x;
    if (i < n)
        w[i] = static_cast<float>(sqrt(s[i]));
}

unsigned blocks_for(int64_t n)
{
    return static_cast<unsigned>((n + kThreads - 1) / kThreads);
}

}  // namespace

extern "C" {

int uqt_div_rn32(const float* a, const float* b, float* q, int64_t n, void* stream)
{
    if (!a || !b || !q || n < 1 || n > (int64_t(1) << 30))
        return -1;
    hipLaunchKernelGGL(k_div, dim3(blocks_for(n)), dim3(kThreads), 0, static_cast<hipStream_t>(stream), a, b, q, n);
    return hipGetLastError() == hipSuccess ? 0 : -5;
}

int uqt_sqrt_rn32(const double* s, float* w, int64_t n, void* stream)
{
    if (!s || !w || n < 1 || n > (int64_t(1) << 30))
        return -1;
    hipLaunchKernelGGL(k_sqrt, dim3(blocks_for(n)), dim3(kThreads), 0, static_cast<hipStream_t>(stream), s, w, n);
    return hipGetLastError() == hipSuccess ? 0 : -5;
}

}  // extern "C"
