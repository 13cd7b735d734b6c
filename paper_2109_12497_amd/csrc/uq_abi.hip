// C ABI of libuq: argument checks on the host, then asynchronous launches.
// Every check completes before the first HIP runtime call, so an invalid
// call returns its status without touching the device or the runtime.
#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>

#include "uq.h"
#include "uq_launch.hpp"

namespace {

thread_local char g_last_error[512] = "";

int fail(int status, const char* fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    std::vsnprintf(g_last_error, sizeof g_last_error, fmt, ap);
    va_end(ap);
    return status;
}

int ok()
{
    g_last_error[0] = '\0';
    return UQ_OK;
}

bool aligned(const void* p, uintptr_t a)
{
    return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0;
}

constexpr int64_t kMaxRows = 65535;           // grid y-dimension
constexpr int64_t kMaxElems = int64_t(1) << 62;

bool integral(float s)
{
    return std::isfinite(s) && std::floor(s) == s;
}

uq::ScaleSet one_scale(float s)
{
    uq::ScaleSet S;
    std::memset(&S, 0, sizeof S);
    S.s[0] = s;
    S.K = 1;
    S.s_last = s;
    return S;
}

int check_scales(const float* scales, int32_t K, uq::ScaleSet* S)
{
    if (K < 1 || K > UQ_MAX_SCALES)
        return fail(UQ_ERANGE, "K = %d is outside [1, %d]", K, UQ_MAX_SCALES);
    if (scales == nullptr)
        return fail(UQ_EINVAL, "scales is NULL");
    std::memset(S, 0, sizeof *S);
    for (int32_t k = 0; k < K; ++k) {
        const float s = scales[k];
        if (!integral(s) || s < 1.0f)
            return fail(UQ_ERANGE, "scales[%d] = %g is not an integer >= 1", k, (double)s);
        if (k > 0 && !(s > scales[k - 1]))
            return fail(UQ_ERANGE, "scales must be strictly increasing (scales[%d] = %g)", k, (double)s);
        S->s[k] = s;
    }
    if (scales[0] > 127.0f)
        return fail(UQ_ERANGE, "smallest scale %g exceeds 127 (codes are int8)", (double)scales[0]);
    S->K = K;
    S->s_last = scales[K - 1];
    return UQ_OK;
}

// M * s exactly representable in binary32 (finite, at most 24 significant bits).
bool exact_product(int32_t M, float s)
{
    int e = 0;
    const double frac = std::frexp(static_cast<double>(s), &e);   // s = frac * 2^e, frac in [0.5, 1)
    uint64_t mant = static_cast<uint64_t>(std::ldexp(frac, 24));  // integral: s has <= 24 bits
    uint64_t prod = static_cast<uint64_t>(M) * mant;
    while (prod != 0 && (prod & 1u) == 0)
        prod >>= 1;
    return prod < (uint64_t(1) << 24) &&
           static_cast<double>(M) * static_cast<double>(s) <= 3.4028234663852886e+38;
}

int check_rows(const void* p, int64_t d, int64_t rows, int64_t ld, int64_t ld_mult, const char* name)
{
    if (p == nullptr && d > 0)
        return fail(UQ_EINVAL, "%s is NULL", name);
    if (ld < d)
        return fail(UQ_EINVAL, "leading dimension of %s (%lld) is smaller than d (%lld)", name,
                    (long long)ld, (long long)d);
    if (ld % ld_mult != 0)
        return fail(UQ_EALIGN, "leading dimension of %s (%lld) is not a multiple of %lld", name,
                    (long long)ld, (long long)ld_mult);
    if (!aligned(p, 16))
        return fail(UQ_EALIGN, "%s is not 16-byte aligned", name);
    if (ld > 0 && rows > kMaxElems / ld)
        return fail(UQ_EINVAL, "%s: rows * leading dimension overflows", name);
    return UQ_OK;
}

int check_vec(const void* p, int64_t d, const char* name)
{
    if (p == nullptr && d > 0)
        return fail(UQ_EINVAL, "%s is NULL", name);
    if (!aligned(p, 16))
        return fail(UQ_EALIGN, "%s is not 16-byte aligned", name);
    return UQ_OK;
}

int check_w(const float* w)
{
    if (w == nullptr)
        return fail(UQ_EINVAL, "w is NULL");
    if (!aligned(w, 4))
        return fail(UQ_EALIGN, "w is not 4-byte aligned");
    return UQ_OK;
}

int check_dims(int64_t d, int64_t rows, const char* rows_name)
{
    if (d < 0 || d > kMaxElems)
        return fail(UQ_EINVAL, "d = %lld is out of range", (long long)d);
    if (rows < 1 || rows > kMaxRows)
        return fail(rows < 1 ? UQ_EINVAL : UQ_ERANGE, "%s = %lld is outside [1, %lld]", rows_name,
                    (long long)rows, (long long)kMaxRows);
    return UQ_OK;
}

int launched(hipError_t e)
{
    if (e != hipSuccess)
        return fail(UQ_EHIP, "HIP launch failed: %s", hipGetErrorString(e));
    return ok();
}

#define UQ_TRY(expr)                  \
    do {                              \
        const int uq_rc_ = (expr);    \
        if (uq_rc_ != UQ_OK)          \
            return uq_rc_;            \
    } while (0)

// The sum's arguments (bits = 8: int8 codes, ld in bytes >= d; 4 or 2:
// packed rows of ceil(d * bits / 8) bytes).
int check_sum(const void* codes, int64_t d, int32_t rows, int64_t ld, int32_t bits, int32_t accumulate,
              const int32_t* sum)
{
    if (d < 0 || d > kMaxElems)
        return fail(UQ_EINVAL, "d = %lld is out of range", (long long)d);
    if (rows < 1)
        return fail(UQ_EINVAL, "rows = %d is smaller than 1", rows);
    if (rows > (1 << 24))
        return fail(UQ_ERANGE, "rows = %d exceeds 2^24 (int32 sums could overflow)", rows);
    if (accumulate != 0 && accumulate != 1)
        return fail(UQ_EINVAL, "accumulate must be 0 or 1");
    UQ_TRY(check_rows(codes, bits == 8 ? d : (d * bits + 7) / 8, rows, ld, 16, bits == 8 ? "codes" : "packed"));
    return check_vec(sum, d, "sum");
}

// The reconstruction's arguments (d already checked); fills *S.
int check_reconstruction(int64_t d, int32_t M, const float* w, const float* scales, int32_t K, const uint8_t* idx,
                         const float* out, uq::ScaleSet* S)
{
    if (M < 1)
        return fail(UQ_EINVAL, "M = %d is smaller than 1", M);
    UQ_TRY(check_scales(scales, K, S));
    if ((K == 1) != (idx == nullptr))
        return fail(UQ_EINVAL, "idx must be NULL exactly when K == 1");
    for (int32_t k = 0; k < K; ++k)
        if (!exact_product(M, S->s[k]))
            return fail(UQ_ERANGE, "M * scales[%d] = %d * %g is not exact in fp32", k, M, (double)S->s[k]);
    if (static_cast<double>(M) * S->s[0] >= 2147483648.0)
        return fail(UQ_ERANGE, "M * s_0 >= 2^31 (int32 sums could overflow)");
    UQ_TRY(check_vec(out, d, "out"));
    UQ_TRY(check_w(w));
    if (K > 1)
        UQ_TRY(check_vec(idx, d > 0 ? d : 1, "idx"));
    return UQ_OK;
}

}  // namespace

namespace uq {

// 64 blocks per compute unit of the current device (the count is cached per
// device; concurrent first calls may both query it and store the same value).
int64_t grid_cap()
{
    static std::atomic<int> cus_by_device[64] = {};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64)
        return 256 * 64;
    int cus = cus_by_device[dev].load(std::memory_order_relaxed);
    if (cus == 0) {
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
            cus = 256;
        cus_by_device[dev].store(cus, std::memory_order_relaxed);
    }
    return static_cast<int64_t>(cus) * 64;
}

}  // namespace uq

namespace {

// Scratch of uq_shared_scale_noalloc: the norm's partial sums (and, with
// several scales and 2 to 16 rows, the rows' maxima) live in this array
// instead of a caller's workspace.  Each device holds its own copy, at its
// own address, until the process ends.  In host code `scratch` names a
// host-side stand-in, never the device memory: kernels get the address that
// hipGetSymbolAddress returns for the current device.
static __device__ __align__(256) unsigned char scratch[UQ_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void* g_scratch_ptr[kMaxDevices] = {};

// The current device's copy of `scratch` (looked up on the first call on
// that device); nullptr with *err set when the runtime refuses.
void* device_scratch(hipError_t* err)
{
    int dev = -1;
    *err = hipGetDevice(&dev);
    if (*err != hipSuccess)
        return nullptr;
    if (dev < 0 || dev >= kMaxDevices) {
        *err = hipErrorInvalidDevice;
        return nullptr;
    }
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (g_scratch_ptr[dev] == nullptr) {
        void* p = nullptr;
        *err = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (*err != hipSuccess)
            return nullptr;
        g_scratch_ptr[dev] = p;
    }
    return g_scratch_ptr[dev];
}

// Scratch bytes uq_shared_scale's kernels use for (d, M, K): the norm's
// partials, or the fused pass's layout.
size_t scratch_bytes_for(int64_t d, int32_t M, int32_t K)
{
    if (uq::use_fused(d, M, K))
        return uq::fused_layout(d, M).bytes;
    const uq::NormPlan p = uq::norm_plan(d);
    const int64_t chunks = p.nchunks < 1 ? 1 : p.nchunks;
    return uq::align256(static_cast<size_t>(M) * static_cast<size_t>(chunks) * sizeof(double));
}

}  // namespace

extern "C" {

size_t uq_workspace_bytes(int64_t d, int32_t M)
{
    const int64_t dd = d < 0 ? 0 : d;
    const uq::NormPlan p = uq::norm_plan(dd);
    const int64_t rows = M < 1 ? 1 : M;
    const int64_t chunks = p.nchunks < 1 ? 1 : p.nchunks;
    size_t bytes = uq::align256(static_cast<size_t>(rows) * static_cast<size_t>(chunks) * sizeof(double));
    // enough for any K: with several scales and few rows the fused pass
    // also keeps the rows' maxima
    if (uq::use_fused(dd, static_cast<int32_t>(rows), 2)) {
        const size_t fused = uq::fused_layout(dd, static_cast<int32_t>(rows)).bytes;
        bytes = fused > bytes ? fused : bytes;
    }
    return bytes;
}

static int shared_scale_common(const float* g, int64_t d, int32_t M, int64_t ldg, const float* scales, int32_t K,
                               float* w, uint8_t* idx, void* ws, size_t ws_bytes, void* stream, int32_t idx_bits)
{
    UQ_TRY(check_dims(d, M, "M"));
    UQ_TRY(check_rows(g, d, M, ldg, 4, "g"));
    UQ_TRY(check_w(w));
    uq::ScaleSet S;
    if (K == 1 && scales == nullptr) {
        S = one_scale(1.0f);
    } else {
        UQ_TRY(check_scales(scales, K, &S));
    }
    if (K > 1)
        UQ_TRY(check_vec(idx, d > 0 ? d : 1, "idx"));
    if (ws == nullptr)
        return fail(UQ_EINVAL, "ws is NULL");
    if (!aligned(ws, 16))
        return fail(UQ_EALIGN, "ws is not 16-byte aligned");
    if (ws_bytes < uq_workspace_bytes(d, M))
        return fail(UQ_EWORKSPACE, "workspace of %zu bytes is smaller than the %zu needed", ws_bytes,
                    uq_workspace_bytes(d, M));
    return launched(
        uq::launch_shared_scale(g, d, M, ldg, S, w, idx, ws, static_cast<hipStream_t>(stream), idx_bits));
}

int uq_shared_scale(const float* g, int64_t d, int32_t M, int64_t ldg, const float* scales, int32_t K,
                    float* w, uint8_t* idx, void* ws, size_t ws_bytes, void* stream)
{
    return shared_scale_common(g, d, M, ldg, scales, K, w, idx, ws, ws_bytes, stream, 8);
}

int uq_shared_scale_idx4(const float* g, int64_t d, int32_t M, int64_t ldg, const float* scales, int32_t K,
                         float* w, uint8_t* idx4, void* ws, size_t ws_bytes, void* stream)
{
    if (K < 2)
        return fail(UQ_EINVAL, "K = %d: the 4-bit index needs several scales", K);
    return shared_scale_common(g, d, M, ldg, scales, K, w, idx4, ws, ws_bytes, stream, 4);
}

int uq_shared_scale_noalloc(const float* g, int64_t d, int32_t M, int64_t ldg, const float* scales, int32_t K,
                            float* w, uint8_t* idx, void* stream)
{
    UQ_TRY(check_dims(d, M, "M"));
    UQ_TRY(check_rows(g, d, M, ldg, 4, "g"));
    UQ_TRY(check_w(w));
    uq::ScaleSet S;
    if (K == 1 && scales == nullptr) {
        S = one_scale(1.0f);
    } else {
        UQ_TRY(check_scales(scales, K, &S));
    }
    if (K > 1)
        UQ_TRY(check_vec(idx, d > 0 ? d : 1, "idx"));
    const size_t need = scratch_bytes_for(d, M, K);
    if (need > UQ_NOALLOC_SCRATCH_BYTES)
        return fail(UQ_EWORKSPACE, "d = %lld, M = %d, K = %d needs %zu bytes of scratch, more than the %zu of the "
                    "static buffer (use uq_shared_scale with a workspace)", (long long)d, M, K, need,
                    (size_t)UQ_NOALLOC_SCRATCH_BYTES);
    hipError_t e = hipSuccess;
    void* ws = device_scratch(&e);
    if (ws == nullptr)
        return fail(UQ_EHIP, "static scratch of the current device: %s", hipGetErrorString(e));
    return launched(uq::launch_shared_scale(g, d, M, ldg, S, w, idx, ws, static_cast<hipStream_t>(stream)));
}

static int quantise_common(const float* g, int64_t d, int32_t rows, int64_t ldg, int32_t worker0,
                           const float* w, const uq::ScaleSet& S, const uint8_t* idx, uint64_t seed,
                           void* codes, int64_t ldc, int32_t bits, void* stream)
{
    UQ_TRY(check_dims(d, rows, "rows"));
    UQ_TRY(check_rows(g, d, rows, ldg, 4, "g"));
    const int64_t row_bytes = (d * bits + 7) / 8;
    UQ_TRY(check_rows(codes, row_bytes, rows, ldc, 16, "codes"));
    UQ_TRY(check_w(w));
    if (worker0 < 0 || static_cast<int64_t>(worker0) + rows > (int64_t(1) << 31))
        return fail(UQ_ERANGE, "worker ids %d .. %lld exceed [0, 2^31)", worker0,
                    (long long)worker0 + rows - 1);
    if (S.K > 1)
        UQ_TRY(check_vec(idx, d > 0 ? d : 1, "idx"));
    return launched(uq::launch_quantise(g, d, rows, ldg, worker0, w, S, idx, seed, codes, ldc, bits,
                                        static_cast<hipStream_t>(stream)));
}

int uq_quantize_single(const float* g, int64_t d, int32_t rows, int64_t ldg, int32_t worker0, const float* w,
                       int32_t s, uint64_t seed, int8_t* codes, int64_t ldc, void* stream)
{
    if (s < 1 || s > 127)
        return fail(UQ_ERANGE, "s = %d is outside [1, 127]", s);
    const uq::ScaleSet S = one_scale(static_cast<float>(s));
    return quantise_common(g, d, rows, ldg, worker0, w, S, nullptr, seed, codes, ldc, 8, stream);
}

int uq_quantize_multi(const float* g, int64_t d, int32_t rows, int64_t ldg, int32_t worker0, const float* w,
                      const float* scales, int32_t K, const uint8_t* idx, uint64_t seed, int8_t* codes,
                      int64_t ldc, void* stream)
{
    uq::ScaleSet S;
    UQ_TRY(check_scales(scales, K, &S));
    if (K > 1 && idx == nullptr && d > 0)
        return fail(UQ_EINVAL, "idx is NULL");
    return quantise_common(g, d, rows, ldg, worker0, w, S, idx, seed, codes, ldc, 8, stream);
}

int uq_quantize_packed(const float* g, int64_t d, int32_t rows, int64_t ldg, int32_t worker0, const float* w,
                       const float* scales, int32_t K, const uint8_t* idx, uint64_t seed, int32_t bits,
                       uint8_t* packed, int64_t ldp, void* stream)
{
    if (bits != 4 && bits != 2)
        return fail(UQ_ERANGE, "bits = %d is not 4 or 2", bits);
    uq::ScaleSet S;
    UQ_TRY(check_scales(scales, K, &S));
    if (S.s[0] > static_cast<float>((1 << (bits - 1)) - 1))
        return fail(UQ_ERANGE, "smallest scale %g does not fit a %d-bit code", (double)S.s[0], bits);
    if (K > 1 && idx == nullptr && d > 0)
        return fail(UQ_EINVAL, "idx is NULL");
    return quantise_common(g, d, rows, ldg, worker0, w, S, idx, seed, packed, ldp, bits, stream);
}

int uq_sum_packed(const uint8_t* packed, int64_t d, int32_t rows, int64_t ldp, int32_t bits, int32_t accumulate,
                  int32_t* sum, void* stream)
{
    if (bits != 4 && bits != 2)
        return fail(UQ_ERANGE, "bits = %d is not 4 or 2", bits);
    UQ_TRY(check_sum(packed, d, rows, ldp, bits, accumulate, sum));
    return launched(uq::launch_sum_packed(packed, d, rows, ldp, bits, accumulate, sum,
                                          static_cast<hipStream_t>(stream)));
}

int uq_sum_codes(const int8_t* codes, int64_t d, int32_t rows, int64_t ldc, int32_t accumulate, int32_t* sum,
                 void* stream)
{
    UQ_TRY(check_sum(codes, d, rows, ldc, 8, accumulate, sum));
    return launched(uq::launch_sum(codes, d, rows, ldc, accumulate, sum, static_cast<hipStream_t>(stream)));
}

int uq_dequantize(const int32_t* sum, int64_t d, int32_t M, const float* w, const float* scales, int32_t K,
                  const uint8_t* idx, float* out, void* stream)
{
    if (d < 0 || d > kMaxElems)
        return fail(UQ_EINVAL, "d = %lld is out of range", (long long)d);
    UQ_TRY(check_vec(sum, d, "sum"));
    uq::ScaleSet S;
    UQ_TRY(check_reconstruction(d, M, w, scales, K, idx, out, &S));
    return launched(uq::launch_dequant(sum, d, M, w, S, idx, out, static_cast<hipStream_t>(stream)));
}

int uq_sum_dequantize(const uint8_t* codes, int64_t d, int32_t rows, int64_t ldc, int32_t bits, int32_t accumulate,
                      int32_t* sum, int32_t M, const float* w, const float* scales, int32_t K, const uint8_t* idx,
                      float* out, void* stream)
{
    if (bits != 8 && bits != 4 && bits != 2)
        return fail(UQ_ERANGE, "bits = %d is not 8, 4 or 2", bits);
    UQ_TRY(check_sum(codes, d, rows, ldc, bits, accumulate, sum));
    uq::ScaleSet S;
    UQ_TRY(check_reconstruction(d, M, w, scales, K, idx, out, &S));
    return launched(uq::launch_sum_dequant(codes, d, rows, ldc, bits, accumulate, sum, M, w, S, idx, out,
                                           static_cast<hipStream_t>(stream)));
}

static int quantize_sum_common(const float* g, int64_t d, int32_t rows, int64_t ldg, int32_t worker0,
                               const float* w, const float* scales, int32_t K, const uint8_t* idx, uint64_t seed,
                               int32_t accumulate, int32_t* sum, int32_t M, float* out, void* stream,
                               int32_t idx_bits)
{
    uq::ScaleSet S;
    UQ_TRY(check_scales(scales, K, &S));
    UQ_TRY(check_dims(d, rows, "rows"));
    UQ_TRY(check_rows(g, d, rows, ldg, 4, "g"));
    UQ_TRY(check_w(w));
    if (worker0 < 0 || static_cast<int64_t>(worker0) + rows > (int64_t(1) << 31))
        return fail(UQ_ERANGE, "worker ids %d .. %lld exceed [0, 2^31)", worker0,
                    (long long)worker0 + rows - 1);
    if (K > 1) {
        if (idx == nullptr && d > 0)
            return fail(UQ_EINVAL, "idx is NULL");
        UQ_TRY(check_vec(idx, d > 0 ? d : 1, "idx"));
    } else {
        idx = nullptr;  // one scale: the index is not read
    }
    if (accumulate != 0 && accumulate != 1)
        return fail(UQ_EINVAL, "accumulate must be 0 or 1");
    UQ_TRY(check_vec(sum, d, "sum"));
    if (out != nullptr) {
        uq::ScaleSet S2;
        UQ_TRY(check_reconstruction(d, M, w, scales, K, idx, out, &S2));
    }
    return launched(uq::launch_quant_sum(g, d, rows, ldg, worker0, w, S, idx, seed, accumulate, sum, M, out,
                                         static_cast<hipStream_t>(stream), idx_bits));
}

int uq_quantize_sum(const float* g, int64_t d, int32_t rows, int64_t ldg, int32_t worker0, const float* w,
                    const float* scales, int32_t K, const uint8_t* idx, uint64_t seed, int32_t accumulate,
                    int32_t* sum, int32_t M, float* out, void* stream)
{
    return quantize_sum_common(g, d, rows, ldg, worker0, w, scales, K, idx, seed, accumulate, sum, M, out, stream,
                               8);
}

int uq_quantize_sum_idx4(const float* g, int64_t d, int32_t rows, int64_t ldg, int32_t worker0, const float* w,
                         const float* scales, int32_t K, const uint8_t* idx4, uint64_t seed, int32_t accumulate,
                         int32_t* sum, int32_t M, float* out, void* stream)
{
    if (K < 2)
        return fail(UQ_EINVAL, "K = %d: the 4-bit index needs several scales", K);
    return quantize_sum_common(g, d, rows, ldg, worker0, w, scales, K, idx4, seed, accumulate, sum, M, out, stream,
                               4);
}

int uq_index_quantize_sum(const float* g, int64_t d, int32_t M, int64_t ldg, const float* w, const float* scales,
                          int32_t K, uint64_t seed, uint8_t* idx, int32_t* sum, float* out, void* stream)
{
    uq::ScaleSet S;
    UQ_TRY(check_scales(scales, K, &S));
    UQ_TRY(check_dims(d, M, "M"));
    if (M > uq::kFuseRows)
        return fail(UQ_ERANGE, "M = %d exceeds the %d rows held in registers", M, uq::kFuseRows);
    UQ_TRY(check_rows(g, d, M, ldg, 4, "g"));
    UQ_TRY(check_w(w));
    if (idx == nullptr && d > 0)
        return fail(UQ_EINVAL, "idx is NULL");
    UQ_TRY(check_vec(idx, d > 0 ? d : 1, "idx"));
    UQ_TRY(check_vec(sum, d, "sum"));
    uq::ScaleSet S2;
    UQ_TRY(check_reconstruction(d, M, w, scales, K, K > 1 ? idx : nullptr, out, &S2));
    return launched(uq::launch_index_quant_sum(g, d, M, ldg, w, S, seed, idx, sum, out,
                                               static_cast<hipStream_t>(stream)));
}

int uq_index_quantize(const float* g, int64_t d, int32_t M, int64_t ldg, const float* w, const float* scales,
                      int32_t K, uint64_t seed, int32_t bits, uint8_t* idx, void* codes, int64_t ldc, void* stream)
{
    if (bits != 8 && bits != 4 && bits != 2)
        return fail(UQ_ERANGE, "bits = %d is not 8, 4 or 2", bits);
    uq::ScaleSet S;
    UQ_TRY(check_scales(scales, K, &S));
    if (bits < 8 && S.s[0] > static_cast<float>((1 << (bits - 1)) - 1))
        return fail(UQ_ERANGE, "smallest scale %g does not fit a %d-bit code", (double)S.s[0], bits);
    UQ_TRY(check_dims(d, M, "M"));
    if (M > uq::kFuseRows)
        return fail(UQ_ERANGE, "M = %d exceeds the %d rows held in registers", M, uq::kFuseRows);
    UQ_TRY(check_rows(g, d, M, ldg, 4, "g"));
    const int64_t row_bytes = (d * bits + 7) / 8;
    UQ_TRY(check_rows(codes, row_bytes, M, ldc, 16, "codes"));
    UQ_TRY(check_w(w));
    if (idx == nullptr && d > 0)
        return fail(UQ_EINVAL, "idx is NULL");
    UQ_TRY(check_vec(idx, d > 0 ? d : 1, "idx"));
    return launched(uq::launch_index_quantise(g, d, M, ldg, w, S, seed, bits, idx, static_cast<uint8_t*>(codes), ldc,
                                              static_cast<hipStream_t>(stream)));
}

size_t uq_randk_workspace_bytes(int64_t d, int64_t K)
{
    (void)d;
    (void)K;
    return uq::randk_workspace_bytes();
}

int uq_randk_select(int64_t d, int64_t K, uint64_t seed, uint32_t* sel, void* ws, size_t ws_bytes, void* stream)
{
    if (d < 1 || d >= (int64_t(1) << 32))
        return fail(UQ_EINVAL, "d = %lld is outside [1, 2^32)", (long long)d);
    if (K < 1 || K > d)
        return fail(UQ_ERANGE, "K = %lld is outside [1, d]", (long long)K);
    UQ_TRY(check_vec(sel, K, "sel"));
    if (ws == nullptr)
        return fail(UQ_EINVAL, "ws is NULL");
    if (!aligned(ws, 16))
        return fail(UQ_EALIGN, "ws is not 16-byte aligned");
    if (ws_bytes < uq_randk_workspace_bytes(d, K))
        return fail(UQ_EWORKSPACE, "workspace of %zu bytes is smaller than the %zu needed", ws_bytes,
                    uq_randk_workspace_bytes(d, K));
    return launched(uq::launch_randk_select(d, K, seed, sel, ws, static_cast<hipStream_t>(stream)));
}

int uq_gather(const float* g, int64_t d, int32_t M, int64_t ldg, const uint32_t* sel, int64_t K, float* sub,
              int64_t lds, void* stream)
{
    UQ_TRY(check_dims(d, M, "M"));
    if (K < 1 || K > d)
        return fail(UQ_ERANGE, "K = %lld is outside [1, d]", (long long)K);
    UQ_TRY(check_rows(g, d, M, ldg, 1, "g"));
    UQ_TRY(check_rows(sub, K, M, lds, 4, "sub"));
    UQ_TRY(check_vec(sel, K, "sel"));
    return launched(uq::launch_gather(g, d, M, ldg, sel, K, sub, lds, static_cast<hipStream_t>(stream)));
}

int uq_scatter(const float* vals, const uint32_t* sel, int64_t K, float* out, int64_t d, void* stream)
{
    if (d < 1 || d > kMaxElems)
        return fail(UQ_EINVAL, "d = %lld is out of range", (long long)d);
    if (K < 1 || K > d)
        return fail(UQ_ERANGE, "K = %lld is outside [1, d]", (long long)K);
    UQ_TRY(check_vec(vals, K, "vals"));
    UQ_TRY(check_vec(sel, K, "sel"));
    UQ_TRY(check_vec(out, d, "out"));
    return launched(uq::launch_scatter(vals, sel, K, out, d, static_cast<hipStream_t>(stream)));
}

int uq_set_randk_mode(int32_t mode)
{
    if (!uq::set_randk_mode(mode))
        return fail(UQ_EINVAL, "GlobalRandK mode %d is not 0, 1, 2, 3 or 4", mode);
    return ok();
}

int uq_set_grid_cap(int64_t blocks)
{
    if (!uq::set_one_shot_cap(blocks))
        return fail(UQ_EINVAL, "grid cap %lld is outside [%lld, 2^22] (0 restores the default)",
                    (long long)blocks, (long long)uq::kMinOneShotCap);
    return ok();
}

const char* uq_strerror(int status)
{
    switch (status) {
    case UQ_OK: return "success";
    case UQ_EINVAL: return "invalid argument";
    case UQ_ERANGE: return "argument out of range";
    case UQ_EALIGN: return "misaligned pointer or leading dimension";
    case UQ_EWORKSPACE: return "workspace too small";
    case UQ_EHIP: return "HIP runtime error";
    default: return "unknown status";
    }
}

const char* uq_last_error(void)
{
    return g_last_error;
}

}  // extern "C"
